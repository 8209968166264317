// Batched full-depth pass over many positions: the prompt pass and the
// periodic refresh of recent positions. The decode program handles one
// position per step and streams every weight once per position; here a
// chunk of positions goes through each layer together, so each weight is
// read once per chunk and the work is a tiled matrix product (positions x
// weight rows) instead of matrix-vector products.
//
// Per layer, five launches (stream order is the only synchronisation):
//   1. QKV:    Y = RMSNorm(X; g_attn) W_qkv^T, RoPE on q and k at each
//              position, k and v stored to the paged cache, q kept;
//   2. attn:   causal grouped-query attention of the chunk's queries over
//              every cached position up to their own (split over key
//              ranges when the chunk alone does not fill the device, then
//              merged in split order);
//   3. W_o:    X += O W_o^T;
//   4. gate/up: A = SiLU(RMSNorm(X; g_mlp) W_g^T) * (RMSNorm(X; g_mlp) W_u^T);
//   5. down:   X += A W_d^T.
// The matrix products split K over several workgroups when the output tiles
// alone do not fill the device; the last workgroup to finish a tile adds the
// K-slices' partial sums in slice order and applies the epilogue, so every
// result is independent of scheduling.
//
// Numerics follow the decode program: weights as stored (bf16 or fp32),
// activations and accumulation fp32, cache entries rounded to the storage
// type (round to nearest even), RMSNorm as x * rsqrt(mean(x^2) + eps) * g
// (the row's scale is applied to the finished dot products), e^x in the
// softmax and SiLU on the hardware base-2 exponential.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "ee_internal.h"

namespace ee {

namespace {

// ---------------------------------------------------------------------------
// helpers (this file's own; the decode kernels keep theirs)
// ---------------------------------------------------------------------------
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent2(float* p, float a, float b) {  // p 8-byte aligned
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p),
                     static_cast<uint64_t>(__float_as_uint(a)) | (static_cast<uint64_t>(__float_as_uint(b)) << 32),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_agent2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<uint64_t*>(const_cast<float*>(p)), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float(static_cast<uint32_t>(v)), __uint_as_float(static_cast<uint32_t>(v >> 32)));
}
__device__ __forceinline__ void drain_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ float exp_hw(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }

template <typename WT>
struct St;

template <>
struct St<uint16_t> {  // bf16 bit patterns
  static constexpr int N = 8;
  __device__ static inline void unpack(const uint4& w, float* f) {
    f[0] = __uint_as_float(w.x << 16);
    f[1] = __uint_as_float(w.x & 0xffff0000u);
    f[2] = __uint_as_float(w.y << 16);
    f[3] = __uint_as_float(w.y & 0xffff0000u);
    f[4] = __uint_as_float(w.z << 16);
    f[5] = __uint_as_float(w.z & 0xffff0000u);
    f[6] = __uint_as_float(w.w << 16);
    f[7] = __uint_as_float(w.w & 0xffff0000u);
  }
  __device__ static inline uint32_t bits(float x) {  // round to nearest even
    uint32_t u = __float_as_uint(x);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
  }
  __device__ static inline void store_pair(uint16_t* p, float a, float b) {
    *reinterpret_cast<uint32_t*>(p) = bits(a) | (bits(b) << 16);
  }
  __device__ static inline float2 load_pair(const uint16_t* p) {
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
  }
};

template <>
struct St<float> {
  static constexpr int N = 4;
  __device__ static inline void unpack(const uint4& w, float* f) {
    f[0] = __uint_as_float(w.x);
    f[1] = __uint_as_float(w.y);
    f[2] = __uint_as_float(w.z);
    f[3] = __uint_as_float(w.w);
  }
  __device__ static inline void store_pair(float* p, float a, float b) {
    *reinterpret_cast<float2*>(p) = make_float2(a, b);
  }
  __device__ static inline float2 load_pair(const float* p) { return *reinterpret_cast<const float2*>(p); }
};

__device__ __forceinline__ int64_t cache_off(const int32_t* block_table, int page_shift, int page_size, int K,
                                             int D, int64_t layer_base, int pos, int kvh) {
  const int page = block_table[pos >> page_shift];
  const int slot = pos & (page_size - 1);
  return layer_base + ((static_cast<int64_t>(page) * K + kvh) * page_size + slot) * D;
}

__device__ __forceinline__ float wave_max64(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace

// ---------------------------------------------------------------------------
// embedding rows of the chunk's tokens
// ---------------------------------------------------------------------------
template <typename WT>
__global__ __launch_bounds__(256) void k_bp_embed(const WT* __restrict__ E, const int32_t* __restrict__ tok, int P,
                                                  int H, int V, float* __restrict__ X, int32_t* hist, int pos0,
                                                  StepCtl* ctl) {
  const int p = blockIdx.x;
  if (p >= P) return;
  int t = tok[p];
  if (t < 0 || t >= V) {
    if (threadIdx.x == 0) atomicMax(&ctl->error, kErrToken);
    t = 0;
  }
  if (threadIdx.x == 0 && hist) hist[pos0 + p] = t;
  const WT* row = E + static_cast<int64_t>(t) * H;
  for (int i0 = 0; i0 < H; i0 += 8 * 256) {
    WT v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + threadIdx.x + 256 * u;
      v[u] = i < H ? row[i] : WT(0);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + threadIdx.x + 256 * u;
      if (i >= H) continue;
      float f;
      if constexpr (sizeof(WT) == 2) f = __uint_as_float(static_cast<uint32_t>(v[u]) << 16);
      else f = v[u];
      X[static_cast<int64_t>(p) * H + i] = f;
    }
  }
}

// ---------------------------------------------------------------------------
// tiled matrix product Y[P][N] = A[P][K] W[N][K]^T with fused RMSNorm of A
// (when gain is set) and an epilogue. Block tile BM positions x BN weight
// rows, 256 threads, each TM x 4 outputs; K in stages of BK (one 128-byte
// line of a weight row), the next stage's tiles loaded into registers while
// the current one is consumed from LDS.
// ---------------------------------------------------------------------------
enum : int { kEpiQkv = 0, kEpiResid = 1, kEpiSwiGlu = 2 };

struct GemmArgs {
  const float* A;      // [P][K] fp32
  const void* W;       // [N][K] storage type
  int P, N, K;
  int k_split;         // K elements per split (multiple of BK), splits = gridDim.z
  const float* gain;   // RMSNorm gain [K] (A is the raw residual stream) or null
  float eps;
  float* part;         // split partials [splits][P][N], then [splits][P] sums of squares
  uint32_t* tile_ctr;  // arrivals per output tile (zero before, reset by the last arrival)
  // epilogue targets
  float* Y;            // kEpiResid: X [P][N] (+=); kEpiSwiGlu: A [P][N/2]; kEpiQkv: q [P][A*D]
  // kEpiQkv: RoPE and cache
  int pos0, Aq, Kh, D;
  const float* rope_cos;
  const float* rope_sin;
  void* kpool;
  void* vpool;
  int64_t layer_base;
  const int32_t* block_table;
  int page_shift, page_size;
};

template <typename WT>
__device__ __forceinline__ void epi_pair(const GemmArgs& g, int EPI, int m, int n, float y0, float y1) {
  if (EPI == kEpiResid) {
    float2* x = reinterpret_cast<float2*>(g.Y + static_cast<int64_t>(m) * g.N + n);
    float2 v = *x;
    v.x += y0;
    v.y += y1;
    *x = v;
  } else if (EPI == kEpiSwiGlu) {
    // interleaved rows: n = 2j gate row j, n + 1 up row j
    const float s = y0 / (1.f + exp_hw(-y0));
    g.Y[static_cast<int64_t>(m) * (g.N >> 1) + (n >> 1)] = s * y1;
  } else {
    // rows of the repacked QKV matrix: q heads, k heads (RoPE pairs
    // interleaved: row 2i = dim i, row 2i+1 = dim i + D/2), v heads
    const int AD = g.Aq * g.D, KD = g.Kh * g.D;
    const int pos = g.pos0 + m;
    if (n < AD + KD) {
      const int head = n / g.D, rl = n - head * g.D, half = g.D >> 1;
      const float c = g.rope_cos[static_cast<int64_t>(pos) * half + (rl >> 1)];
      const float s = g.rope_sin[static_cast<int64_t>(pos) * half + (rl >> 1)];
      const float r0 = y0 * c - y1 * s;
      const float r1 = y1 * c + y0 * s;
      if (n < AD) {
        *reinterpret_cast<float2*>(g.Y + static_cast<int64_t>(m) * AD + n) = make_float2(r0, r1);
      } else {
        const int64_t off = cache_off(g.block_table, g.page_shift, g.page_size, g.Kh, g.D, g.layer_base, pos,
                                      head - g.Aq);
        St<WT>::store_pair(static_cast<WT*>(g.kpool) + off + rl, r0, r1);
      }
    } else {
      const int j = n - AD - KD;
      const int head = j / g.D, d = j - head * g.D;
      const int64_t off = cache_off(g.block_table, g.page_shift, g.page_size, g.Kh, g.D, g.layer_base, pos, head);
      St<WT>::store_pair(static_cast<WT*>(g.vpool) + off + d, y0, y1);
    }
  }
}

template <typename WT, int EPI, int BM, int BN, int TM>
__global__ __launch_bounds__(256) void k_bp_gemm(GemmArgs g) {
  constexpr int TN = 4;
  constexpr int EPC = St<WT>::N;           // elements per 16-byte chunk
  constexpr int BK = 128 / sizeof(WT);     // one 128-byte line of a weight row per stage
  constexpr int CPR = BK / EPC;            // chunks per row per stage (8)
  constexpr int TX = BN / TN;              // threads along N
  static_assert((BM / TM) * TX == 256, "256 threads");
  constexpr int WCH = BN * CPR / 256;      // weight chunks per thread per stage
  constexpr int AQ = BM * BK / 4;          // float4 of A per stage
  constexpr int ACH = (AQ + 255) / 256;    // float4 per thread per stage
  constexpr int LW = BN + 4;               // LDS row strides (floats)
  constexpr int LA = BM + 4;
  __shared__ float Ws[BK * LW];
  __shared__ float As[BK * LA];
  __shared__ float ss_part[BM];
  __shared__ int last_flag;

  const int tid = threadIdx.x;
  const int tx = tid % TX, ty = tid / TX;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const int split = blockIdx.z, splits = gridDim.z;
  const int kb = split * g.k_split, ke = min(g.K, kb + g.k_split);
  const WT* W = static_cast<const WT*>(g.W);

  uint4 wr[WCH];
  float4 ar[ACH];
  float ssq[ACH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) ssq[i] = 0.f;

  auto load_stage = [&](int k0) {
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      const int c = tid + 256 * i;
      const int r = c / CPR, q = c - r * CPR;
      const int n = n0 + r, k = k0 + q * EPC;
      wr[i] = (n < g.N && k < ke) ? *reinterpret_cast<const uint4*>(W + static_cast<int64_t>(n) * g.K + k)
                                  : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + 256 * i;
      const int m = c / (BK / 4), q = c - m * (BK / 4);
      const int k = k0 + 4 * q;
      ar[i] = (c < AQ && m0 + m < g.P && k < ke)
                  ? *reinterpret_cast<const float4*>(g.A + static_cast<int64_t>(m0 + m) * g.K + k)
                  : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store_stage = [&](int k0) {
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      const int c = tid + 256 * i;
      const int r = c / CPR, q = c - r * CPR;
      float f[EPC];
      St<WT>::unpack(wr[i], f);
#pragma unroll
      for (int e = 0; e < EPC; ++e) Ws[(q * EPC + e) * LW + r] = f[e];
    }
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + 256 * i;
      if (c < AQ) {
        const int m = c / (BK / 4), q = c - m * (BK / 4);
        const int k = k0 + 4 * q;
        float4 a = ar[i];
        if (g.gain) {
          ssq[i] = fmaf(a.x, a.x, fmaf(a.y, a.y, fmaf(a.z, a.z, fmaf(a.w, a.w, ssq[i]))));
          if (k < ke) {
            const float4 gg = *reinterpret_cast<const float4*>(g.gain + k);
            a.x *= gg.x; a.y *= gg.y; a.z *= gg.z; a.w *= gg.w;
          }
        }
        As[(4 * q + 0) * LA + m] = a.x;
        As[(4 * q + 1) * LA + m] = a.y;
        As[(4 * q + 2) * LA + m] = a.z;
        As[(4 * q + 3) * LA + m] = a.w;
      }
    }
  };

  float acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = 0.f;

  if (kb < ke) load_stage(kb);
  for (int k0 = kb; k0 < ke; k0 += BK) {
    __syncthreads();
    store_stage(k0);
    __syncthreads();
    if (k0 + BK < ke) load_stage(k0 + BK);
#pragma unroll 8
    for (int k = 0; k < BK; ++k) {
      float a[TM];
      if constexpr (TM == 4) {
        const float4 av = *reinterpret_cast<const float4*>(&As[k * LA + ty * TM]);
        a[0] = av.x; a[1] = av.y; a[2] = av.z; a[3] = av.w;
      } else {
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = As[k * LA + ty * TM + i];
      }
      const float4 wv = *reinterpret_cast<const float4*>(&Ws[k * LW + tx * TN]);
      const float w[TN] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
  }

  // per-row sums of squares of this K-slice: the BK/4 threads of a row are
  // consecutive lanes; the first of them holds the row's sum
  if (g.gain) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      float v = ssq[i];
#pragma unroll
      for (int o = 1; o < BK / 4; o <<= 1) v += __shfl_xor(v, o);
      const int c = tid + 256 * i;
      if (c < AQ && (c % (BK / 4)) == 0) ss_part[c / (BK / 4)] = v;
    }
  }
  __syncthreads();

  const int64_t PN = static_cast<int64_t>(g.P) * g.N;
  if (splits > 1) {
    // publish this slice's partial tile; the last arrival merges all slices
    float* part = g.part + split * PN;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + ty * TM + i;
      if (m >= g.P) continue;
#pragma unroll
      for (int j = 0; j < TN; j += 2) {
        const int n = n0 + tx * TN + j;
        if (n < g.N) st_agent2(part + static_cast<int64_t>(m) * g.N + n, acc[i][j], acc[i][j + 1]);
      }
    }
    if (g.gain && tid < BM && m0 + tid < g.P) st_agent(g.part + splits * PN + split * g.P + m0 + tid, ss_part[tid]);
    drain_stores();
    __syncthreads();
    if (tid == 0) {
      uint32_t* ctr = g.tile_ctr + blockIdx.y * gridDim.x + blockIdx.x;
      const uint32_t old = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last_flag = old == static_cast<uint32_t>(splits - 1);
      if (last_flag) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!last_flag) return;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = 0.f;
    // the slices' partial sums in slice order; each group of kSG slices has
    // all its loads in flight before the first is added
    constexpr int kSG = TM >= 4 ? 2 : 8;  // 16 pairs in flight per thread
    for (int s0 = 0; s0 < splits; s0 += kSG) {
      float2 v[kSG][TM][TN / 2];
#pragma unroll
      for (int u = 0; u < kSG; ++u) {
        const float* ps = g.part + (s0 + u) * PN;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int m = m0 + ty * TM + i;
#pragma unroll
          for (int j = 0; j < TN; j += 2) {
            const int n = n0 + tx * TN + j;
            v[u][i][j / 2] = (s0 + u < splits && m < g.P && n < g.N)
                                 ? ld_agent2(ps + static_cast<int64_t>(m) * g.N + n)
                                 : make_float2(0.f, 0.f);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kSG; ++u)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; j += 2) {
            acc[i][j] += v[u][i][j / 2].x;
            acc[i][j + 1] += v[u][i][j / 2].y;
          }
    }
    if (g.gain && tid < BM && m0 + tid < g.P) {
      float t = 0.f;
      for (int s0 = 0; s0 < splits; s0 += kSG) {
        float v[kSG];
#pragma unroll
        for (int u = 0; u < kSG; ++u)
          v[u] = s0 + u < splits ? ld_agent(g.part + splits * PN + (s0 + u) * g.P + m0 + tid) : 0.f;
#pragma unroll
        for (int u = 0; u < kSG; ++u) t += v[u];
      }
      ss_part[tid] = t;
    }
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int ml = ty * TM + i, m = m0 + ml;
    if (m >= g.P) continue;
    const float rinv = g.gain ? rsqrtf(ss_part[ml] / static_cast<float>(g.K) + g.eps) : 1.f;
#pragma unroll
    for (int j = 0; j < TN; j += 2) {
      const int n = n0 + tx * TN + j;
      if (n < g.N) epi_pair<WT>(g, EPI, m, n, acc[i][j] * rinv, acc[i][j + 1] * rinv);
    }
  }
}

// ---------------------------------------------------------------------------
// causal grouped-query attention of a chunk of queries (positions pos0 ..
// pos0 + P - 1) over the cache. Block = (KV head, tile of 4 query
// positions, key split); wave w takes query position 4 t + w with the G query
// heads of the KV head; keys in tiles of 64 staged in LDS, lane j = key j of
// the tile; online softmax per head. One split writes o directly; several
// write partial records (weighted V, max, sum) merged in split order by
// k_bp_attn_merge.
// ---------------------------------------------------------------------------
struct AttnArgs {
  const float* Q;      // [P][A*D], pair-interleaved within heads (as the cached keys)
  float* O;            // [P][A*D], natural order
  float* part;         // [P][A][nsplit][D + 2]
  const void* kpool;
  const void* vpool;
  int64_t layer_base;
  const int32_t* block_table;
  int page_shift, page_size;
  int P, pos0, A, K, G, D;
  int nsplit, keys_per_split;
  float scale;
};

constexpr int kQT = 4;   // query positions per block (one per wave)
constexpr int kKT = 64;  // keys per LDS tile

template <typename WT, int D>
__global__ __launch_bounds__(256) void k_bp_attn(AttnArgs a) {
  constexpr int EPC = St<WT>::N;
  constexpr int CPK = D / EPC;          // 16-byte chunks per cache row
  constexpr int DPL = D / 64;           // output dimensions per lane (1 or 2)
  constexpr int KST = CPK + 1;          // key rows padded by one chunk: lane j reads row j
  __shared__ uint4 Ks[kKT * KST];
  __shared__ uint4 Vs[kKT * CPK];
  __shared__ float Qs[kQT][kMaxGroup][D];
  __shared__ float Ps[kQT][kMaxGroup][kKT];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nqt = (a.P + kQT - 1) / kQT;
  const int item = blockIdx.x;
  const int kvh = item / (nqt * a.nsplit);
  const int rem = item - kvh * nqt * a.nsplit;
  const int qt = rem / a.nsplit, sp = rem - qt * a.nsplit;
  const int G = a.G;
  const int qi = qt * kQT + wave;               // query index within the chunk
  const bool active = qi < a.P;
  const int qpos = a.pos0 + qi;                 // its position
  const int t_end = a.pos0 + min(a.P, (qt + 1) * kQT);  // keys needed by the tile: [0, t_end)
  const int kb = sp * a.keys_per_split;
  const int ke = min(t_end, kb + a.keys_per_split);

  // the wave's query rows (G heads of this KV head), every load in flight at once
  {
    constexpr int QPL = kMaxGroup * D / 64;
    float qv[QPL];
#pragma unroll
    for (int u = 0; u < QPL; ++u) {
      const int i = lane + 64 * u, h = i / D, d = i - h * D;
      qv[u] = (active && h < G) ? a.Q[static_cast<int64_t>(qi) * a.A * D + (kvh * G + h) * D + d] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < QPL; ++u) {
      const int i = lane + 64 * u, h = i / D, d = i - h * D;
      Qs[wave][h][d] = qv[u];
    }
  }
  float m_run[kMaxGroup], l_run[kMaxGroup], acc[kMaxGroup][DPL];
#pragma unroll
  for (int h = 0; h < kMaxGroup; ++h) {
    m_run[h] = -INFINITY;
    l_run[h] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[h][e] = 0.f;
  }
  const WT* kp = static_cast<const WT*>(a.kpool);
  const WT* vp = static_cast<const WT*>(a.vpool);

  constexpr int CPT = kKT * CPK / 256;  // chunks of K (and of V) per thread per tile
  for (int k0 = kb; k0 < ke; k0 += kKT) {
    // every page lookup of the tile, then every K and V load, before any
    // result is waited for: two round trips per tile
    int64_t off[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i;
      const int j = c / CPK, q = c - j * CPK;
      const int key = min(k0 + j, ke - 1);
      off[i] = cache_off(a.block_table, a.page_shift, a.page_size, a.K, D, a.layer_base, key, kvh) + q * EPC;
    }
    uint4 kv[CPT], vv[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      kv[i] = *reinterpret_cast<const uint4*>(kp + off[i]);
      vv[i] = *reinterpret_cast<const uint4*>(vp + off[i]);
    }
    __syncthreads();  // previous tile consumed (and Qs written before the first)
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i;
      const int j = c / CPK, q = c - j * CPK;
      Ks[j * KST + q] = kv[i];  // keys past ke repeat key ke - 1; their scores are masked
      Vs[c] = vv[i];
    }
    __syncthreads();
    const int key = k0 + lane;
    const bool valid = active && key < ke && key <= qpos;
    float s[kMaxGroup];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) s[h] = 0.f;
#pragma unroll 4
    for (int q = 0; q < CPK; ++q) {
      float kf[EPC];
      St<WT>::unpack(Ks[lane * KST + q], kf);
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        if (h < G) {
#pragma unroll
          for (int e = 0; e < EPC; ++e) s[h] = fmaf(Qs[wave][h][q * EPC + e], kf[e], s[h]);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      if (h >= G) continue;
      const float sv = valid ? s[h] * a.scale : -INFINITY;
      const float mt = wave_max64(sv);
      const float mn = fmaxf(m_run[h], mt);
      float p = 0.f, alpha = 1.f;
      if (mn != -INFINITY) {
        p = exp_hw(sv - mn);  // 0 for masked keys
        alpha = exp_hw(m_run[h] - mn);
      }
      l_run[h] = l_run[h] * alpha + wave_sum64(p);
      m_run[h] = mn;
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[h][e] *= alpha;
      Ps[wave][h][lane] = p;
    }
    __builtin_amdgcn_wave_barrier();
    // weighted values: lane owns dimensions DPL * lane .. + DPL - 1
#pragma unroll 8
    for (int j = 0; j < kKT; ++j) {
      float v[DPL];
      if constexpr (DPL == 2) {
        const float2 vv = St<WT>::load_pair(reinterpret_cast<const WT*>(&Vs[j * CPK]) + 2 * lane);
        v[0] = vv.x;
        v[1] = vv.y;
      } else {
        const WT* vr = reinterpret_cast<const WT*>(&Vs[j * CPK]);
        if constexpr (sizeof(WT) == 2) v[0] = __uint_as_float(static_cast<uint32_t>(vr[lane]) << 16);
        else v[0] = vr[lane];
      }
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        if (h < G) {
          const float pj = Ps[wave][h][j];
#pragma unroll
          for (int e = 0; e < DPL; ++e) acc[h][e] = fmaf(pj, v[e], acc[h][e]);
        }
      }
    }
  }
  if (!active) return;
#pragma unroll
  for (int h = 0; h < kMaxGroup; ++h) {
    if (h >= G) continue;
    const int head = kvh * G + h;
    if (a.nsplit == 1) {
      const float inv = 1.f / l_run[h];
#pragma unroll
      for (int e = 0; e < DPL; ++e)
        a.O[static_cast<int64_t>(qi) * a.A * D + head * D + DPL * lane + e] = acc[h][e] * inv;
    } else {
      float* r = a.part + ((static_cast<int64_t>(qi) * a.A + head) * a.nsplit + sp) * (D + 2);
#pragma unroll
      for (int e = 0; e < DPL; ++e) r[DPL * lane + e] = acc[h][e];
      if (lane == 0) {
        r[D] = m_run[h];
        r[D + 1] = l_run[h];
      }
    }
  }
}

// one wave per (query, head): the splits' partial records in split order
template <int D>
__global__ __launch_bounds__(256) void k_bp_attn_merge(AttnArgs a) {
  constexpr int DPL = D / 64;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (w >= a.P * a.A) return;
  const float* r = a.part + static_cast<int64_t>(w) * a.nsplit * (D + 2);
  float M = -INFINITY;
  float den = 0.f, num[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) num[e] = 0.f;
  // groups of 8 splits: every record of a group requested before any is used
  constexpr int kSG = 8;
  for (int s0 = 0; s0 < a.nsplit; s0 += kSG) {
    float ms[kSG], ls[kSG], vs[kSG][DPL];
#pragma unroll
    for (int u = 0; u < kSG; ++u) {
      const bool ok = s0 + u < a.nsplit;
      const float* q = r + (s0 + u) * (D + 2);
      ms[u] = ok ? q[D] : -INFINITY;
      ls[u] = ok ? q[D + 1] : 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) vs[u][e] = ok ? q[DPL * lane + e] : 0.f;
    }
    // running maximum over the splits so far, in split order
    float cm = M;
#pragma unroll
    for (int u = 0; u < kSG; ++u) cm = fmaxf(cm, ms[u]);
    if (cm != -INFINITY) {
      const float sc = exp_hw(M - cm);  // 0 while nothing has been merged
      den *= sc;
#pragma unroll
      for (int e = 0; e < DPL; ++e) num[e] *= sc;
#pragma unroll
      for (int u = 0; u < kSG; ++u) {
        if (ms[u] == -INFINITY) continue;  // absent, or a split wholly past the query's position
        const float f = exp_hw(ms[u] - cm);
        den = fmaf(f, ls[u], den);
#pragma unroll
        for (int e = 0; e < DPL; ++e) num[e] = fmaf(f, vs[u][e], num[e]);
      }
      M = cm;
    }
  }
  const int qi = w / a.A, head = w - qi * a.A;
  const float inv = 1.f / den;
#pragma unroll
  for (int e = 0; e < DPL; ++e) a.O[static_cast<int64_t>(qi) * a.A * D + head * D + DPL * lane + e] = num[e] * inv;
}

// ---------------------------------------------------------------------------
// host driver
// ---------------------------------------------------------------------------
namespace {

// Splits of K so that the grid holds at least ~2 workgroups per compute unit,
// bounded by the partial workspace and by one stage per split.
void choose_split(int tiles, int P, int N, int K, int BK, size_t ws_floats, int wgs_per_cu, int n_cu, int* k_split,
                  int* splits) {
  // enough workgroups per compute unit (wgs_per_cu) that their weight loads
  // in flight together cover the memory latency; at most 32 slices
  int s = std::max(1, (wgs_per_cu * n_cu + tiles - 1) / tiles);
  s = std::min({s, (K + BK - 1) / BK, 32});
  const size_t per = static_cast<size_t>(P) * N + P;
  if (per > 0) s = static_cast<int>(std::min<size_t>(s, std::max<size_t>(1, ws_floats / per)));
  if (s <= 1) {
    *k_split = K;
    *splits = 1;
    return;
  }
  int ks = (K + s - 1) / s;
  ks = (ks + BK - 1) / BK * BK;
  *k_split = ks;
  *splits = (K + ks - 1) / ks;
}

template <typename WT, int EPI>
hipError_t gemm(const GemmArgs& g0, const BatchBuffers& b, int n_cu, hipStream_t s) {
  GemmArgs g = g0;
  constexpr int BK = 128 / sizeof(WT);
  if (g.P <= 16) {
    // few positions: narrow tiles (16 positions x 64 rows, one position and
    // four rows per thread) so that few K-slices fill the device and the
    // merge of a tile's slices stays short
    constexpr int BM = 16, BN = 64, TM = 1;
    const int tiles = ((g.N + BN - 1) / BN) * ((g.P + BM - 1) / BM);
    int splits;
    // a tile of 16 positions does little arithmetic per weight byte: many
    // short K-slices, so that loads of several workgroups per unit overlap
    choose_split(tiles, g.P, g.N, g.K, BK, b.gemm_ws_floats, 8, n_cu, &g.k_split, &splits);
    if (static_cast<size_t>(tiles) > b.n_tile_ctr) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_bp_gemm<WT, EPI, BM, BN, TM>), dim3((g.N + BN - 1) / BN, (g.P + BM - 1) / BM, splits),
                       dim3(256), 0, s, g);
  } else {
    constexpr int BM = 64, BN = 64, TM = 4;
    const int tiles = ((g.N + BN - 1) / BN) * ((g.P + BM - 1) / BM);
    int splits;
    choose_split(tiles, g.P, g.N, g.K, BK, b.gemm_ws_floats, 2, n_cu, &g.k_split, &splits);
    if (static_cast<size_t>(tiles) > b.n_tile_ctr) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_bp_gemm<WT, EPI, BM, BN, TM>), dim3((g.N + BN - 1) / BN, (g.P + BM - 1) / BM, splits),
                       dim3(256), 0, s, g);
  }
  return hipGetLastError();
}

template <typename WT, int D>
hipError_t attention(AttnArgs a, const BatchBuffers& b, int n_cu, hipStream_t s) {
  const int nqt = (a.P + kQT - 1) / kQT;
  const int t_max = a.pos0 + a.P;
  const int key_tiles = (t_max + kKT - 1) / kKT;
  int ns = std::max(1, (4 * n_cu + a.K * nqt - 1) / (a.K * nqt));
  ns = std::min(ns, key_tiles);
  const size_t per = static_cast<size_t>(a.P) * a.A * (D + 2);
  ns = static_cast<int>(std::min<size_t>(ns, std::max<size_t>(1, b.attn_ws_floats / per)));
  a.keys_per_split = (key_tiles + ns - 1) / ns * kKT;
  a.nsplit = (t_max + a.keys_per_split - 1) / a.keys_per_split;
  hipLaunchKernelGGL((k_bp_attn<WT, D>), dim3(a.K * nqt * a.nsplit), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nsplit == 1) return e;
  hipLaunchKernelGGL((k_bp_attn_merge<D>), dim3((a.P * a.A + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <typename WT>
hipError_t attention_d(const AttnArgs& a, const BatchBuffers& b, int n_cu, hipStream_t s) {
  switch (a.D) {
    case 32: return hipErrorInvalidValue;  // rows of at least 64 dimensions (one per lane)
    case 64: return attention<WT, 64>(a, b, n_cu, s);
    case 128: return attention<WT, 128>(a, b, n_cu, s);
  }
  return hipErrorInvalidValue;
}

template <typename WT>
hipError_t pass(const BatchPass& bp, int pos0, const int32_t* d_tokens, int n, hipStream_t s) {
  const DevParams& p = bp.p;
  const BatchBuffers& b = bp.buf;
  hipError_t e;
  for (int c0 = 0; c0 < n; c0 += b.max_positions) {
    const int P = std::min(b.max_positions, n - c0);
    const int cpos = pos0 + c0;
    hipLaunchKernelGGL((k_bp_embed<WT>), dim3(P), dim3(256), 0, s, static_cast<const WT*>(p.embed), d_tokens + c0, P,
                       p.H, p.V, b.X, p.hist_tok, cpos, p.ctl);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    for (int l = 0; l < p.L; ++l) {
      const LayerW& lw = bp.layers[l];
      GemmArgs g{};
      g.P = P;
      g.eps = p.eps;
      g.part = b.gemm_ws;
      g.tile_ctr = b.tile_ctr;
      g.pos0 = cpos;
      g.Aq = p.A;
      g.Kh = p.K;
      g.D = p.D;
      g.rope_cos = p.rope_cos;
      g.rope_sin = p.rope_sin;
      g.kpool = p.kpool;
      g.vpool = p.vpool;
      g.layer_base = static_cast<int64_t>(l) * p.layer_stride;
      g.block_table = p.block_table;
      g.page_shift = p.page_shift;
      g.page_size = p.page_size;
      // 1. QKV with the attention RMSNorm, RoPE and the cache stores
      GemmArgs q = g;
      q.A = b.X; q.W = lw.wqkv; q.N = p.qkv_rows; q.K = p.H; q.gain = lw.g_attn; q.Y = b.Q;
      if ((e = gemm<WT, kEpiQkv>(q, b, bp.n_cu, s)) != hipSuccess) return e;
      // 2. attention over every cached position up to each query's own
      AttnArgs at{};
      at.Q = b.Q; at.O = b.O; at.part = b.attn_ws;
      at.kpool = p.kpool; at.vpool = p.vpool; at.layer_base = g.layer_base;
      at.block_table = p.block_table; at.page_shift = p.page_shift; at.page_size = p.page_size;
      at.P = P; at.pos0 = cpos; at.A = p.A; at.K = p.K; at.G = p.G; at.D = p.D; at.scale = p.attn_scale;
      if ((e = attention_d<WT>(at, b, bp.n_cu, s)) != hipSuccess) return e;
      // 3. X += O W_o^T
      GemmArgs o = g;
      o.A = b.O; o.W = lw.wo; o.N = p.H; o.K = p.A * p.D; o.gain = nullptr; o.Y = b.X;
      if ((e = gemm<WT, kEpiResid>(o, b, bp.n_cu, s)) != hipSuccess) return e;
      // 4. SiLU(gate) * up with the feed-forward RMSNorm
      GemmArgs gu = g;
      gu.A = b.X; gu.W = lw.wgu; gu.N = 2 * p.F; gu.K = p.H; gu.gain = lw.g_mlp; gu.Y = b.Act;
      if ((e = gemm<WT, kEpiSwiGlu>(gu, b, bp.n_cu, s)) != hipSuccess) return e;
      // 5. X += A W_d^T
      GemmArgs dn = g;
      dn.A = b.Act; dn.W = lw.wd; dn.N = p.H; dn.K = p.F; dn.gain = nullptr; dn.Y = b.X;
      if ((e = gemm<WT, kEpiResid>(dn, b, bp.n_cu, s)) != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_batched_pass(const BatchPass& bp, int pos0, const int32_t* d_tokens, int n, hipStream_t s) {
  if (n <= 0 || bp.buf.max_positions <= 0) return hipErrorInvalidValue;
  return bp.wbf16 ? pass<uint16_t>(bp, pos0, d_tokens, n, s) : pass<float>(bp, pos0, d_tokens, n, s);
}

size_t batch_tile_counters(int max_positions, int N_max) {
  // tiles of 64 x 64 (more than 16 positions) and 16 x 64 (at most 16)
  const size_t a = static_cast<size_t>((N_max + 63) / 64) * ((max_positions + 63) / 64);
  const size_t b = static_cast<size_t>((N_max + 63) / 64);
  return std::max(a, b);
}

}  // namespace ee
