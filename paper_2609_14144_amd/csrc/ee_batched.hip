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

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

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

// Bounds-checked 16-byte loads without a branch: an out-of-range lane reads
// from `safe` (any valid address) and its bits are masked to zero where the
// value is consumed. A load inside a conditional, or selected against zero,
// is compiled to a branch around the load, and the branch's join waits for
// every outstanding load; masking at the load itself waits for the load
// there. Either would serialise a ring of prefetches.
template <typename T>
__device__ __forceinline__ T ld_clamped(const T* p, const T* safe, bool ok) {
  return *(ok ? p : safe);
}
template <typename T>
__device__ __forceinline__ T zero_unless(T v, bool ok) {
  static_assert(sizeof(T) == 16, "16-byte values");
  u32x4 u = __builtin_bit_cast(u32x4, v);
  u &= ok ? 0xffffffffu : 0u;
  return __builtin_bit_cast(T, u);
}

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

// Wave reductions: DPP within rows of 16 lanes, then the four row results
// by readlane; every lane gets the same value, summed in a fixed order.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_of(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ float wave_max64(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));   // lane ^ 1
  v = fmaxf(v, dpp_mov<0x4E>(v));   // lane ^ 2
  v = fmaxf(v, dpp_mov<0x141>(v));  // the other quad of the 8
  v = fmaxf(v, dpp_mov<0x140>(v));  // the other 8 of the 16
  return fmaxf(fmaxf(lane_of(v, 0), lane_of(v, 16)), fmaxf(lane_of(v, 32), lane_of(v, 48)));
}
__device__ __forceinline__ float wave_sum64(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x141>(v);
  v += dpp_mov<0x140>(v);
  return (lane_of(v, 0) + lane_of(v, 16)) + (lane_of(v, 32) + lane_of(v, 48));
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
// The same product for bf16 weights on the matrix cores
// (v_mfma_f32_16x16x32_bf16): 16 weight rows x 16 positions per MFMA. The
// weights are exact bf16 operands; every fp32 activation x (times its gain)
// is split exactly into three bf16 terms t1 + t2 + t3 (t1 its top 16 bits,
// t2 those of the remainder, t3 the rest, which fits in 8 significant bits),
// and the three products accumulate in fp32, so the result carries fp32
// accumulation error only, as the vector-ALU product does.
// Block: 4 waves, each RB row blocks of 16 rows; CP column blocks of 16
// positions; K in steps of 64. Lane l (row / position l % 16, group
// g = l / 16) loads 32 contiguous bytes of its row, k0 + 16 g .. + 15 (four
// lanes read a whole 128-byte line); the low half feeds one MFMA whose k
// slots (g, j) are k0 + 16 g + j, the high half a second with k0 + 16 g + 8
// + j, and the activation operands in LDS are laid out to match.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& u) { return __builtin_bit_cast(bf16x8, u); }

// three bf16 terms of each of four floats: term t of element i in 16 bits
__device__ __forceinline__ void split3(const float4& x, uint2* t) {
  const float v[4] = {x.x, x.y, x.z, x.w};
  uint32_t b[3][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t u = __float_as_uint(v[i]);
    const uint32_t h1 = u & 0xffff0000u;
    const float r1 = v[i] - __uint_as_float(h1);
    const uint32_t h2 = __float_as_uint(r1) & 0xffff0000u;
    const float r2 = r1 - __uint_as_float(h2);
    b[0][i] = h1 >> 16;
    b[1][i] = h2 >> 16;
    b[2][i] = __float_as_uint(r2) >> 16;  // exact: r2 has at most 8 significant bits
  }
#pragma unroll
  for (int k = 0; k < 3; ++k) t[k] = make_uint2(b[k][0] | (b[k][1] << 16), b[k][2] | (b[k][3] << 16));
}

// A ring of PF steps of weight and activation loads is in flight; bounds are
// applied without branches (an out-of-range lane reads a valid address and
// is masked where consumed: a branch around a load makes its join wait for
// every outstanding load), and the K-slice's RMSNorm gains are staged in LDS
// once (a gain load per step would be waited for together with the ring).
constexpr int kWideGainMax = 2048;  // longest K-slice of a normalised product on wide tiles

template <int EPI, int RB, int CP, int PF>
__global__ __launch_bounds__(256) void k_bp_gemm_mfma(GemmArgs g) {
  constexpr int BN = 64 * RB, BP = 16 * CP, KS = 64;
  constexpr int XCH = BP * KS / 4 / 256;  // float4 of activations per thread per step
  // activation terms of one step, double buffered:
  // [buf][term][column block][group][position][half] as 16-byte chunks
  __shared__ uint4 Xs[2][3][CP][4][16][2];
  __shared__ float ss_part[BP];
  __shared__ int last_flag;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lg = lane >> 4, lr = lane & 15;
  const int n0 = blockIdx.x * BN, p0 = blockIdx.y * BP;
  const int split = blockIdx.z, splits = gridDim.z;
  const int kb = split * g.k_split, ke = min(g.K, kb + g.k_split);
  const uint16_t* W = static_cast<const uint16_t*>(g.W);

  constexpr int kGW = kWideGainMax / (4 * 256);  // gain float4s per thread
  __shared__ float4 gsm[EPI != kEpiResid ? kWideGainMax / 4 : 1];
  float4 gl[EPI != kEpiResid ? kGW : 1];
  if constexpr (EPI != kEpiResid) {
    const float4* g4 = reinterpret_cast<const float4*>(g.gain + kb);
#pragma unroll
    for (int j = 0; j < kGW; ++j) gl[j] = ld_clamped(g4 + tid + 256 * j, g4, 4 * (tid + 256 * j) < ke - kb);
    asm volatile("" ::: "memory");  // issued before the ring's loads
  }
  float ssq[XCH];
#pragma unroll
  for (int i = 0; i < XCH; ++i) ssq[i] = 0.f;
  const int nsteps = (ke - kb + KS - 1) / KS;
  uint4 wq[PF][RB][2];
  float4 xq[PF][XCH];
  // loads of step st into ring slot `slot` (masked when consumed)
  auto load = [&](int st, int slot) {
    const bool sok = st < nsteps;
    const int k0 = kb + st * KS;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int n = n0 + (wave * RB + rb) * 16 + lr;
      const int k = k0 + 16 * lg;
      const uint4* src = reinterpret_cast<const uint4*>(W + static_cast<int64_t>(n) * g.K + k);
      const uint4* w0 = reinterpret_cast<const uint4*>(W);
      wq[slot][rb][0] = ld_clamped(src, w0, sok && n < g.N && k < ke);
      wq[slot][rb][1] = ld_clamped(src + 1, w0, sok && n < g.N && k + 8 < ke);
    }
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      const int c = tid + 256 * i;
      const int p = c >> 4, k = k0 + 4 * (c & 15);
      xq[slot][i] = ld_clamped(reinterpret_cast<const float4*>(g.A + static_cast<int64_t>(p0 + p) * g.K + k),
                               reinterpret_cast<const float4*>(g.A), sok && p0 + p < g.P && k < ke);
    }
  };
  // step st's activations of ring slot `slot`: masked, normalised, split into
  // three bf16 terms in LDS buffer buf
  auto store_x = [&](int buf, int st, int slot) {
    const int k0 = kb + st * KS;
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      const int c = tid + 256 * i;
      const int p = c >> 4, kq = c & 15, k = k0 + 4 * kq;
      float4 a = zero_unless(xq[slot][i], p0 + p < g.P && k < ke);
      if constexpr (EPI != kEpiResid) {
        ssq[i] = fmaf(a.x, a.x, fmaf(a.y, a.y, fmaf(a.z, a.z, fmaf(a.w, a.w, ssq[i]))));
        const float4 gg = gsm[min(k - kb, kWideGainMax - 4) / 4];
        a.x *= gg.x; a.y *= gg.y; a.z *= gg.z; a.w *= gg.w;
      }
      uint2 t[3];
      split3(a, t);
      const int grp = kq >> 2, j0 = 4 * (kq & 3);  // k - k0 = 16 grp + j0
#pragma unroll
      for (int term = 0; term < 3; ++term) {
        uint2* dst = reinterpret_cast<uint2*>(&Xs[buf][term][p >> 4][grp][p & 15][j0 >> 3]) + ((j0 >> 2) & 1);
        *dst = t[term];
      }
    }
  };

  f32x4 acc[RB][CP];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int cp = 0; cp < CP; ++cp) acc[rb][cp] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto products = [&](int buf, const uint4 (&wc)[RB][2]) {
#pragma unroll
    for (int cp = 0; cp < CP; ++cp) {
#pragma unroll
      for (int term = 0; term < 3; ++term) {
        const bf16x8 blo = as_bf16x8(Xs[buf][term][cp][lg][lr][0]);
        const bf16x8 bhi = as_bf16x8(Xs[buf][term][cp][lg][lr][1]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          acc[rb][cp] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wc[rb][0]), blo, acc[rb][cp], 0, 0, 0);
          acc[rb][cp] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wc[rb][1]), bhi, acc[rb][cp], 0, 0, 0);
        }
      }
    }
  };

#pragma unroll
  for (int i = 0; i < PF; ++i) load(i, i);
  if constexpr (EPI != kEpiResid) {
    asm volatile("" ::: "memory");  // the ring's loads all issued first
    static_assert(kGW * 256 * 4 == kWideGainMax, "gain staging covers the LDS copy");
#pragma unroll
    for (int j = 0; j < kGW; ++j) gsm[tid + 256 * j] = gl[j];  // past the slice: valid gains of masked activations
    __syncthreads();
  }
  int buf = 0;
  for (int st0 = 0; st0 < nsteps; st0 += PF) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int st = st0 + i;
      if (st >= nsteps) break;  // the same for every wave
      store_x(buf, st, i);
      __syncthreads();
      const int k = kb + st * KS + 16 * lg;
      uint4 wc[RB][2];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const bool rok = n0 + (wave * RB + rb) * 16 + lr < g.N;
        wc[rb][0] = zero_unless(wq[i][rb][0], rok && k < ke);
        wc[rb][1] = zero_unless(wq[i][rb][1], rok && k + 8 < ke);
      }
      load(st + PF, i);  // refill the slot just read
      products(buf, wc);
      buf ^= 1;  // the other buffer is written next; this one is read until the barrier after that store
    }
  }

  // per-position sums of squares of this K-slice: the 16 threads of a
  // position are consecutive lanes
  if (g.gain) {
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      float v = ssq[i];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o);
      const int c = tid + 256 * i;
      if ((c & 15) == 0) ss_part[c >> 4] = v;
    }
  }
  __syncthreads();

  // lane's outputs: rows n0 + (wave RB + rb) 16 + 4 lg + i (i < 4), position p0 + 16 cp + lr
  const int64_t PN = static_cast<int64_t>(g.P) * g.N;
  if (splits > 1) {
    float* part = g.part + split * PN;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int cp = 0; cp < CP; ++cp) {
        const int n = n0 + (wave * RB + rb) * 16 + 4 * lg, p = p0 + 16 * cp + lr;
        if (n < g.N && p < g.P) {
          float* d = part + static_cast<int64_t>(p) * g.N + n;
          st_agent2(d, acc[rb][cp][0], acc[rb][cp][1]);
          st_agent2(d + 2, acc[rb][cp][2], acc[rb][cp][3]);
        }
      }
    if (g.gain && tid < BP && p0 + tid < g.P) st_agent(g.part + splits * PN + split * g.P + p0 + tid, ss_part[tid]);
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
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int cp = 0; cp < CP; ++cp) acc[rb][cp] = f32x4{0.f, 0.f, 0.f, 0.f};
    constexpr int kSG = (RB * CP >= 4) ? 1 : 16;  // slices with loads in flight together
    for (int s0 = 0; s0 < splits; s0 += kSG) {
      float2 v[kSG][RB][CP][2];
#pragma unroll
      for (int u = 0; u < kSG; ++u)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int cp = 0; cp < CP; ++cp) {
            const int n = n0 + (wave * RB + rb) * 16 + 4 * lg, p = p0 + 16 * cp + lr;
            const bool ok = s0 + u < splits && n < g.N && p < g.P;
            const float* d = g.part + (s0 + u) * PN + static_cast<int64_t>(p) * g.N + n;
            v[u][rb][cp][0] = ok ? ld_agent2(d) : make_float2(0.f, 0.f);
            v[u][rb][cp][1] = ok ? ld_agent2(d + 2) : make_float2(0.f, 0.f);
          }
#pragma unroll
      for (int u = 0; u < kSG; ++u)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int cp = 0; cp < CP; ++cp) {
            acc[rb][cp][0] += v[u][rb][cp][0].x;
            acc[rb][cp][1] += v[u][rb][cp][0].y;
            acc[rb][cp][2] += v[u][rb][cp][1].x;
            acc[rb][cp][3] += v[u][rb][cp][1].y;
          }
    }
    if (g.gain && tid < BP && p0 + tid < g.P) {
      float t = 0.f;
      for (int s0 = 0; s0 < splits; s0 += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          v[u] = s0 + u < splits ? ld_agent(g.part + splits * PN + (s0 + u) * g.P + p0 + tid) : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u) t += v[u];
      }
      ss_part[tid] = t;
    }
    __syncthreads();
  }

#pragma unroll
  for (int cp = 0; cp < CP; ++cp) {
    const int pl = 16 * cp + lr, p = p0 + pl;
    if (p >= g.P) continue;
    const float rinv = g.gain ? rsqrtf(ss_part[pl] / static_cast<float>(g.K) + g.eps) : 1.f;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int n = n0 + (wave * RB + rb) * 16 + 4 * lg;
      if (n < g.N) epi_pair<uint16_t>(g, EPI, p, n, acc[rb][cp][0] * rinv, acc[rb][cp][1] * rinv);
      if (n + 2 < g.N) epi_pair<uint16_t>(g, EPI, p, n + 2, acc[rb][cp][2] * rinv, acc[rb][cp][3] * rinv);
    }
  }
}

// ---------------------------------------------------------------------------
// Few positions (P <= 16) on the matrix cores: a workgroup owns RB x 16
// weight rows and all 16 positions over one K-slice (blockIdx.y of
// gridDim.y), its NW waves split the slice into contiguous ranges of 64-wide
// steps, and the waves' sums meet in LDS in wave order. Lane l (row /
// position l % 16, group l / 16) loads its own operands straight into
// registers: 32 bytes of its weight row and 16 activations of its position,
// the same k range k0 + 16 (l / 16) .. + 15 as above (the slice's RMSNorm
// gains come from LDS); a ring of PF steps is in flight. With several slices
// the last workgroup of a tile to arrive adds the slices' sums (and sums of
// squares) in slice order.
// ---------------------------------------------------------------------------
constexpr int kNarrowGainMax = 4096;  // longest K-slice of a normalised product on narrow tiles

template <int EPI, int RB, int NW, int PF>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_bp_gemm_narrow(GemmArgs g) {
  constexpr int KS = 64;
  constexpr bool kGain = EPI != kEpiResid;  // the gated products normalise their input
  constexpr int kGQ = kNarrowGainMax / (4 * NW * 64);  // gain float4s per thread
  __shared__ f32x4 red[NW][RB][64];
  __shared__ float ssr[NW][64];
  __shared__ float4 gs[kGain ? kNarrowGainMax / 4 : 1];  // the slice's RMSNorm gains
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lg = lane >> 4, lr = lane & 15;
  const int n0 = blockIdx.x * 16 * RB;
  const int split = blockIdx.y, splits = gridDim.y;
  const int kb = split * g.k_split, ke = min(g.K, kb + g.k_split);
  const int nsteps = (ke - kb + KS - 1) / KS;
  const int s0 = nsteps * wave / NW, s1 = nsteps * (wave + 1) / NW;
  // every wave runs the same number of ring turns (steps at or past s1
  // read a valid address and are masked to zero), so that the loop body
  // has no branch: a branch around a load makes its join wait for every
  // outstanding load
  const int turns = ((nsteps + NW - 1) / NW + PF - 1) / PF;
  const bool pok = lr < g.P;
  const uint16_t* W = static_cast<const uint16_t*>(g.W);
  const float* xrow = g.A + static_cast<int64_t>(lr) * g.K;

  // the slice's gains go through LDS (they are the same for every row and
  // position); their loads are issued ahead of the weight ring's
  float4 gl[kGain ? kGQ : 1];
  if constexpr (kGain) {
    const float4* g4 = reinterpret_cast<const float4*>(g.gain + kb);
#pragma unroll
    for (int j = 0; j < kGQ; ++j) {
      const int c = tid + NW * 64 * j;
      gl[j] = ld_clamped(g4 + c, g4, 4 * c < ke - kb);
    }
    // issued before the weight loads (the vector-memory counter is in
    // order), so their LDS copy below waits for them alone
    asm volatile("" ::: "memory");
  }
  uint4 wr[PF][RB][2];
  float4 xr[PF][4];
  // loads of step st into ring slot `slot`, out-of-range parts masked when
  // the slot is consumed
  auto load = [&](int st, int slot) {
    const bool sok = st < s1;
    const int k = kb + st * KS + 16 * lg;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = n0 + rb * 16 + lr;
      const uint4* src = reinterpret_cast<const uint4*>(W + static_cast<int64_t>(row) * g.K + k);
      const uint4* w0 = reinterpret_cast<const uint4*>(W);
      wr[slot][rb][0] = ld_clamped(src, w0, sok && row < g.N && k < ke);
      wr[slot][rb][1] = ld_clamped(src + 1, w0, sok && row < g.N && k + 8 < ke);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
      xr[slot][q] = ld_clamped(reinterpret_cast<const float4*>(xrow + k + 4 * q),
                               reinterpret_cast<const float4*>(g.A), sok && pok && k + 4 * q < ke);
  };
  f32x4 acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float ssq = 0.f;
#pragma unroll
  for (int i = 0; i < PF; ++i) load(s0 + i, i);
  if constexpr (kGain) {
    asm volatile("" ::: "memory");  // the ring's loads all issued first
    static_assert(kGQ * NW * 64 * 4 == kNarrowGainMax, "gain staging covers the LDS copy");
#pragma unroll
    for (int j = 0; j < kGQ; ++j) {
      const int c = tid + NW * 64 * j;
      gs[c] = gl[j];  // past the slice: a valid gain, multiplying masked (zero) activations
    }
    __syncthreads();
  }
  for (int turn = 0; turn < turns; ++turn) {
    const int st0 = s0 + turn * PF;
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      {
        const int st = st0 + i;
        const bool sok = st < s1;
        const int k = kb + st * KS + 16 * lg;
        float4 x[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          x[q] = zero_unless(xr[i][q], sok && pok && k + 4 * q < ke);
          if constexpr (kGain) {
            const float4 gq = gs[min((k - kb) / 4 + q, kNarrowGainMax / 4 - 1)];
            ssq = fmaf(x[q].x, x[q].x, fmaf(x[q].y, x[q].y, fmaf(x[q].z, x[q].z, fmaf(x[q].w, x[q].w, ssq))));
            x[q].x *= gq.x; x[q].y *= gq.y; x[q].z *= gq.z; x[q].w *= gq.w;
          }
        }
        // three bf16 terms of the low (k .. k + 7) and high (k + 8 .. + 15) halves
        uint2 t[4][3];
#pragma unroll
        for (int q = 0; q < 4; ++q) split3(x[q], t[q]);
        uint4 wc[RB][2];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const bool rok = n0 + rb * 16 + lr < g.N;
          wc[rb][0] = zero_unless(wr[i][rb][0], sok && rok && k < ke);
          wc[rb][1] = zero_unless(wr[i][rb][1], sok && rok && k + 8 < ke);
        }
        load(st + PF, i);  // refill the slot just read
#pragma unroll
        for (int term = 0; term < 3; ++term) {
          const uint4 blo = make_uint4(t[0][term].x, t[0][term].y, t[1][term].x, t[1][term].y);
          const uint4 bhi = make_uint4(t[2][term].x, t[2][term].y, t[3][term].x, t[3][term].y);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wc[rb][0]), as_bf16x8(blo), acc[rb], 0, 0, 0);
            acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wc[rb][1]), as_bf16x8(bhi), acc[rb], 0, 0, 0);
          }
        }
      }
    }
  }
  // The tile's outputs in units of two: unit u = (row block u / 2, half
  // u % 2 of each lane's four rows), lane (lg, lr) holding rows
  // n0 + 16 (u / 2) + 4 lg + 2 (u % 2) + {0, 1} of position lr. Wave w sums
  // units w, w + NW, ... over the waves' partial products (in wave order)
  // and, with several K-slices, stores them, and the last workgroup of the
  // tile to arrive merges every slice of every unit with all of its loads in
  // flight at once.
  constexpr int NU = 2 * RB, UPW = (NU + NW - 1) / NW;
  __shared__ int last_flag;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) red[wave][rb][lane] = acc[rb];
  ssr[wave][lane] = ssq;
  __syncthreads();
  float2 y[UPW];
#pragma unroll
  for (int j = 0; j < UPW; ++j) {
    const int u = wave + NW * j;
    y[j] = make_float2(0.f, 0.f);
    if (u < NU) {
      const int rb = u >> 1, c = 2 * (u & 1);
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        y[j].x += red[w][rb][lane][c];
        y[j].y += red[w][rb][lane][c + 1];
      }
    }
  }
  // position lr's sum of squares over the slice: the four lane groups of
  // every wave
  float t = 0.f;
  if constexpr (kGain) {
#pragma unroll
    for (int w = 0; w < NW; ++w)
      t += (ssr[w][lr] + ssr[w][lr + 16]) + (ssr[w][lr + 32] + ssr[w][lr + 48]);
  }
  auto unit_n = [&](int j) { const int u = wave + NW * j; return n0 + 16 * (u >> 1) + 4 * lg + 2 * (u & 1); };
  auto unit_ok = [&](int j) { return wave + NW * j < NU && unit_n(j) < g.N && pok; };
  // the residual rows the epilogue adds to, requested before any wait
  float2 xold[EPI == kEpiResid ? UPW : 1];
  if constexpr (EPI == kEpiResid) {
#pragma unroll
    for (int j = 0; j < UPW; ++j) {
      const float2* xp = reinterpret_cast<const float2*>(g.Y + static_cast<int64_t>(lr) * g.N + unit_n(j));
      xold[j] = unit_ok(j) ? *xp : make_float2(0.f, 0.f);
    }
  }
  if (splits > 1) {
    const int64_t PN = static_cast<int64_t>(g.P) * g.N;
#pragma unroll
    for (int j = 0; j < UPW; ++j)
      if (unit_ok(j)) st_agent2(g.part + split * PN + static_cast<int64_t>(lr) * g.N + unit_n(j), y[j].x, y[j].y);
    if (kGain && wave == 0 && lg == 0 && pok) st_agent(g.part + splits * PN + split * g.P + lr, t);
    drain_stores();
    __syncthreads();  // every wave's partial sums stored
    if (tid == 0) {
      uint32_t* ctr = g.tile_ctr + blockIdx.x;
      const uint32_t old = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last_flag = old == static_cast<uint32_t>(splits - 1);
      if (last_flag) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!last_flag) return;
    constexpr int kSG = 16;  // slices with loads in flight together
#pragma unroll
    for (int j = 0; j < UPW; ++j) y[j] = make_float2(0.f, 0.f);
    t = 0.f;
    for (int q0 = 0; q0 < splits; q0 += kSG) {
      float2 v[UPW][kSG];
      float vs[kSG];
#pragma unroll
      for (int u = 0; u < kSG; ++u) {
#pragma unroll
        for (int j = 0; j < UPW; ++j) {
          const float* d = g.part + (q0 + u) * PN + static_cast<int64_t>(lr) * g.N + unit_n(j);
          v[j][u] = (unit_ok(j) && q0 + u < splits) ? ld_agent2(d) : make_float2(0.f, 0.f);
        }
        vs[u] = (kGain && pok && q0 + u < splits) ? ld_agent(g.part + splits * PN + (q0 + u) * g.P + lr) : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kSG; ++u) {
#pragma unroll
        for (int j = 0; j < UPW; ++j) {
          y[j].x += v[j][u].x;
          y[j].y += v[j][u].y;
        }
        t += vs[u];
      }
    }
  }
  const float rinv = kGain ? rsqrtf(t / static_cast<float>(g.K) + g.eps) : 1.f;
#pragma unroll
  for (int j = 0; j < UPW; ++j) {
    if (!unit_ok(j)) continue;
    const int n = unit_n(j);
    if constexpr (EPI == kEpiResid) {
      *reinterpret_cast<float2*>(g.Y + static_cast<int64_t>(lr) * g.N + n) =
          make_float2(xold[j].x + y[j].x, xold[j].y + y[j].y);
    } else {
      epi_pair<uint16_t>(g, EPI, lr, n, y[j].x * rinv, y[j].y * rinv);
    }
  }
}

// ---------------------------------------------------------------------------
// causal grouped-query attention of a chunk of queries (positions pos0 ..
// pos0 + P - 1) over the cache. Block = (KV head, tile of 4 query
// positions, key split); its waves split the tile's queries and the KV
// head's query heads; keys in tiles of 64 staged in LDS, lane j = key j of
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

constexpr int kKT = 64;  // keys per LDS tile

// Block = (KV head, tile of QT query positions, key split); wave w takes
// query position w % QT and the GW query heads (w / QT) GW .. + GW - 1 of the
// KV head. With many blocks (a prompt) QT = 4 and each wave takes all G heads
// (more waves would read each key tile from LDS once per wave), at most two
// workgroups per compute unit (as LDS allows), so each wave may hold up to
// 256 registers; with few blocks (a refresh) QT = 2 and one head per wave,
// so that the G heads' dot products run on G waves per position. The first
// four waves stage each key tile in LDS.
// (fp32 caches of wide heads may need more registers: their lower bound is 1)
template <typename WT, int D, int G, int GW, int QT>
__global__ __launch_bounds__(64 * QT * (G / GW))
__attribute__((amdgpu_waves_per_eu(sizeof(WT) == 4 ? 1 : ((QT * (G / GW) + 3) / 4 > 2 ? (QT * (G / GW) + 3) / 4 : 2),
                                   (QT * (G / GW) + 3) / 4 > 2 ? (QT * (G / GW) + 3) / 4 : 2))) void k_bp_attn(AttnArgs a) {
  static_assert(G % GW == 0, "head groups cover the KV head's query heads");
  static_assert(QT * (G / GW) >= 4, "four waves stage the key tiles");
  constexpr int kQT = QT;
  constexpr int EPC = St<WT>::N;
  constexpr int CPK = D / EPC;          // 16-byte chunks per cache row
  constexpr int DPL = D / 64;           // output dimensions per lane (1 or 2)
  constexpr int KST = CPK + 1;          // key rows padded by one chunk: lane j reads row j
  __shared__ uint4 Ks[kKT * KST];
  __shared__ uint4 Vs[kKT * CPK];
  __shared__ float Qs[kQT][G][D];
  __shared__ float Ps[kQT][G][kKT];

  constexpr int HG = G / GW;            // waves per query position
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int qw = HG > 1 ? wave % kQT : wave, h0 = HG > 1 ? (wave / kQT) * GW : 0;
  const bool loader = HG > 1 ? tid < 256 : true;  // the threads that stage key tiles
  const int nqt = (a.P + kQT - 1) / kQT;
  const int item = blockIdx.x;
  const int kvh = item / (nqt * a.nsplit);
  const int rem = item - kvh * nqt * a.nsplit;
  const int qt = rem / a.nsplit, sp = rem - qt * a.nsplit;
  const int qi = qt * kQT + qw;                 // query index within the chunk
  const bool active = qi < a.P;
  const int qpos = a.pos0 + qi;                 // its position
  const int t_end = a.pos0 + min(a.P, (qt + 1) * kQT);  // keys needed by the tile: [0, t_end)
  const int kb = sp * a.keys_per_split;
  const int ke = min(t_end, kb + a.keys_per_split);

  constexpr int CPT = kKT * CPK / 256;  // chunks of K (and of V) per loading thread per tile
  // cache offsets of a tile's chunks (its page lookups)
  auto offsets = [&](int k0, int64_t (&off)[CPT]) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i;
      const int j = c / CPK, q = c - j * CPK;
      const int key = min(k0 + j, ke - 1);
      off[i] = cache_off(a.block_table, a.page_shift, a.page_size, a.K, D, a.layer_base, key, kvh) + q * EPC;
    }
  };
  // the wave's query rows (its GW heads) and the first tile's page lookups,
  // every load in flight at once
  int64_t off[CPT];
  if (loader && kb < ke) offsets(kb, off);
  {
    constexpr int QPL = GW * D / 64;
    float qv[QPL];
#pragma unroll
    for (int u = 0; u < QPL; ++u) {
      const int i = lane + 64 * u, h = h0 + i / D, d = i % D;
      qv[u] = active ? a.Q[static_cast<int64_t>(qi) * a.A * D + (kvh * G + h) * D + d] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < QPL; ++u) {
      const int i = lane + 64 * u, h = h0 + i / D, d = i % D;
      Qs[qw][h][d] = qv[u];
    }
  }
  float m_run[GW], l_run[GW], acc[GW][DPL];
#pragma unroll
  for (int h = 0; h < GW; ++h) {
    m_run[h] = -INFINITY;
    l_run[h] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[h][e] = 0.f;
  }
  const WT* kp = static_cast<const WT*>(a.kpool);
  const WT* vp = static_cast<const WT*>(a.vpool);

  for (int k0 = kb; k0 < ke; k0 += kKT) {
    // native vectors: a copy of the uint4 struct from global memory to LDS
    // through registers compiles to memory-to-memory copies through private
    // memory, which serialise the loads
    u32x4 kv[CPT], vv[CPT];
    if (loader) {
      if (k0 != kb) offsets(k0, off);
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        kv[i] = *reinterpret_cast<const u32x4*>(kp + off[i]);
        vv[i] = *reinterpret_cast<const u32x4*>(vp + off[i]);
      }
    }
    __syncthreads();  // previous tile consumed (and Qs written before the first)
    if (loader) {
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int c = tid + 256 * i;
        const int j = c / CPK, q = c - j * CPK;
        *reinterpret_cast<u32x4*>(&Ks[j * KST + q]) = kv[i];  // keys past ke repeat key ke - 1; masked
        *reinterpret_cast<u32x4*>(&Vs[c]) = vv[i];
      }
    }
    __syncthreads();
    const int key = k0 + lane;
    const bool valid = active && key < ke && key <= qpos;
    float s[GW];
#pragma unroll
    for (int h = 0; h < GW; ++h) s[h] = 0.f;
#pragma unroll 2
    for (int q = 0; q < CPK; ++q) {
      float kf[EPC];
      St<WT>::unpack(Ks[lane * KST + q], kf);
#pragma unroll
      for (int h = 0; h < GW; ++h) {
#pragma unroll
        for (int e = 0; e < EPC; ++e) s[h] = fmaf(Qs[qw][h0 + h][q * EPC + e], kf[e], s[h]);
      }
    }
#pragma unroll
    for (int h = 0; h < GW; ++h) {
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
      Ps[qw][h0 + h][lane] = p;
    }
    __builtin_amdgcn_wave_barrier();
    // weighted values: lane owns dimensions DPL * lane .. + DPL - 1
#pragma unroll 4
    for (int j = 0; j < kKT; ++j) {
      float v[DPL];
      if constexpr (DPL == 2) {
        const float2 vv2 = St<WT>::load_pair(reinterpret_cast<const WT*>(&Vs[j * CPK]) + 2 * lane);
        v[0] = vv2.x;
        v[1] = vv2.y;
      } else {
        const WT* vr = reinterpret_cast<const WT*>(&Vs[j * CPK]);
        if constexpr (sizeof(WT) == 2) v[0] = __uint_as_float(static_cast<uint32_t>(vr[lane]) << 16);
        else v[0] = vr[lane];
      }
#pragma unroll
      for (int h = 0; h < GW; ++h) {
        const float pj = Ps[qw][h0 + h][j];
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[h][e] = fmaf(pj, v[e], acc[h][e]);
      }
    }
  }
  if (!active) return;
#pragma unroll
  for (int h = 0; h < GW; ++h) {
    const int head = kvh * G + h0 + h;
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
                  int* splits, int max_k_split = 1 << 30) {
  // enough workgroups per compute unit (wgs_per_cu) that their weight loads
  // in flight together cover the memory latency; at most 32 slices, and
  // slices of at most max_k_split
  int s = std::max(1, (wgs_per_cu * n_cu + tiles - 1) / tiles);
  s = std::max(s, (K + max_k_split - 1) / max_k_split);
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

template <int EPI, int RB, int CP, int PF>
hipError_t gemm_mfma(GemmArgs g, const BatchBuffers& b, int n_cu, int wgs_per_cu, hipStream_t s) {
  constexpr int BN = 64 * RB, BP = 16 * CP;
  const int tiles = ((g.N + BN - 1) / BN) * ((g.P + BP - 1) / BP);
  if (static_cast<size_t>(tiles) > b.n_tile_ctr) return hipErrorInvalidValue;
  int splits;
  choose_split(tiles, g.P, g.N, g.K, 64, b.gemm_ws_floats, wgs_per_cu, n_cu, &g.k_split, &splits,
               EPI != kEpiResid ? kWideGainMax : (1 << 30));
  if (EPI != kEpiResid && g.k_split > kWideGainMax) return hipErrorInvalidValue;  // gains staged in LDS
  hipLaunchKernelGGL((k_bp_gemm_mfma<EPI, RB, CP, PF>), dim3((g.N + BN - 1) / BN, (g.P + BP - 1) / BP, splits),
                     dim3(256), 0, s, g);
  return hipGetLastError();
}

// Narrow tiles for at most 16 positions: RB x 16 rows by NW waves, which
// split each K-slice into contiguous ranges of 64-wide steps. K is split over
// workgroups where the tiles alone leave units idle: tiles times slices stay
// within one round of the units' slots (eight waves per unit), with at least
// two steps per wave.
constexpr int64_t kSliceMergeBytes = 72 << 10;

struct NarrowPlan {
  int tiles, splits, k_split;
  int64_t busiest;  // bytes the busiest unit loads (bf16 weights and 16 fp32 activation rows)
};
NarrowPlan narrow_plan(int EPI, int RB, int NW, const GemmArgs& g, size_t ws_floats, int n_cu,
                       bool whole_k = false) {
  NarrowPlan q;
  q.tiles = (g.N + 16 * RB - 1) / (16 * RB);
  const int slots = n_cu * (8 / NW);
  int splits = whole_k ? 1 : std::max(1, std::min(slots / q.tiles, (g.K + 64 * 2 * NW - 1) / (64 * 2 * NW)));
  if (EPI != kEpiResid) splits = std::max(splits, (g.K + kNarrowGainMax - 1) / kNarrowGainMax);
  const size_t per = static_cast<size_t>(g.P) * g.N + g.P;
  splits = static_cast<int>(std::min<size_t>(splits, std::max<size_t>(1, ws_floats / per)));
  q.k_split = ((g.K + splits - 1) / splits + 63) / 64 * 64;
  q.splits = (g.K + q.k_split - 1) / q.k_split;
  const int64_t wgs = static_cast<int64_t>(q.tiles) * q.splits;
  q.busiest = (wgs + n_cu - 1) / n_cu * static_cast<int64_t>(q.k_split) * (32 * RB + 64);
  // a K-slice merge (partial stores, their drain, the arrival count, the
  // slices' loads: ~3 us) costs about what a unit loads in that time
  if (q.splits > 1) q.busiest += kSliceMergeBytes;
  return q;
}

template <int EPI, int RB, int NW, int PF>
hipError_t gemm_narrow(GemmArgs g, const BatchBuffers& b, int n_cu, hipStream_t s, bool whole_k = false) {
  const NarrowPlan q = narrow_plan(EPI, RB, NW, g, b.gemm_ws_floats, n_cu, whole_k);
  if (static_cast<size_t>(q.tiles) > b.n_tile_ctr) return hipErrorInvalidValue;
  if (EPI != kEpiResid && q.k_split > kNarrowGainMax) return hipErrorInvalidValue;
  g.k_split = q.k_split;
  hipLaunchKernelGGL((k_bp_gemm_narrow<EPI, RB, NW, PF>), dim3(q.tiles, q.splits), dim3(NW * 64), 0, s, g);
  return hipGetLastError();
}

template <typename WT, int EPI>
hipError_t gemm(const GemmArgs& g0, const BatchBuffers& b, int n_cu, hipStream_t s) {
  GemmArgs g = g0;
  constexpr int BK = 128 / sizeof(WT);
  if constexpr (sizeof(WT) == 2) {
    // bf16 weights: matrix cores; 64 rows x 16 positions per workgroup for
    // few positions (many short K-slices keep the weight stream in flight),
    // else 128 rows x 64 positions
    if (g.P <= 16) {
      // few positions: narrow tiles. Large tiles of eight waves (one
      // workgroup per unit) keep most of a matrix in flight at once; small
      // tiles of four waves (two per unit) balance the units where the large
      // tiles would leave some with two. The K split fills the units.
      if constexpr (EPI == kEpiSwiGlu) {
        // 80-row tiles of eight waves, or 64-row tiles of four waves (two
        // per unit): whichever leaves the busiest unit fewer bytes to load
        const NarrowPlan a5 = narrow_plan(EPI, 5, 8, g, b.gemm_ws_floats, n_cu);
        const NarrowPlan a4 = narrow_plan(EPI, 4, 4, g, b.gemm_ws_floats, n_cu);
        if (a4.busiest < a5.busiest) return gemm_narrow<EPI, 4, 4, 2>(g, b, n_cu, s);
        return gemm_narrow<EPI, 5, 8, 2>(g, b, n_cu, s);
      } else if constexpr (EPI == kEpiResid) {
        // 64-row tiles of eight waves or 32-row tiles of four, by the same rule
        const NarrowPlan a4 = narrow_plan(EPI, 4, 8, g, b.gemm_ws_floats, n_cu);
        const NarrowPlan a2 = narrow_plan(EPI, 2, 4, g, b.gemm_ws_floats, n_cu);
        const NarrowPlan a1 = narrow_plan(EPI, 1, 8, g, b.gemm_ws_floats, n_cu, true);
        if (a1.busiest < a2.busiest && a1.busiest < a4.busiest) return gemm_narrow<EPI, 1, 8, 2>(g, b, n_cu, s, true);
        if (a4.busiest < a2.busiest) return gemm_narrow<EPI, 4, 8, 2>(g, b, n_cu, s);
        return gemm_narrow<EPI, 2, 4, 2>(g, b, n_cu, s);
      } else {
        // 32-row tiles of four waves, or 16-row tiles of eight waves over the
        // whole K (no slice merge), by the same rule
        const NarrowPlan a2 = narrow_plan(EPI, 2, 4, g, b.gemm_ws_floats, n_cu);
        const NarrowPlan a1 = narrow_plan(EPI, 1, 8, g, b.gemm_ws_floats, n_cu, true);
        if (a1.busiest < a2.busiest) return gemm_narrow<EPI, 1, 8, 2>(g, b, n_cu, s, true);
        return gemm_narrow<EPI, 2, 4, 2>(g, b, n_cu, s);
      }
    }
    return gemm_mfma<EPI, 2, 4, 3>(g, b, n_cu, 2, s);
  }
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
  constexpr int kQT = 4;  // query positions per block of the prompt's path
  const int nqt = (a.P + kQT - 1) / kQT;
  const int t_max = a.pos0 + a.P;
  const int key_tiles = (t_max + kKT - 1) / kKT;
  int ns = std::max(1, (4 * n_cu + a.K * nqt - 1) / (a.K * nqt));
  ns = std::min(ns, key_tiles);
  const size_t per = static_cast<size_t>(a.P) * a.A * (D + 2);
  ns = static_cast<int>(std::min<size_t>(ns, std::max<size_t>(1, b.attn_ws_floats / per)));
  a.keys_per_split = (key_tiles + ns - 1) / ns * kKT;
  a.nsplit = (t_max + a.keys_per_split - 1) / a.keys_per_split;
  // few blocks: blocks of two query positions whose waves take one query
  // head each; else four positions, one wave each with all heads
  const bool split_heads = static_cast<int64_t>(a.K) * nqt * a.nsplit < 2 * n_cu && a.G >= 2;
  const dim3 grid(a.K * (split_heads ? (a.P + 1) / 2 : nqt) * a.nsplit);
  switch (a.G) {
#define EE_ATTN_G(GG)                                                                                  \
  case GG:                                                                                             \
    if (GG >= 2 && split_heads) {                                                                      \
      hipLaunchKernelGGL((k_bp_attn<WT, D, GG, 1, (GG >= 2 ? 2 : 4)>), grid, dim3(128 * GG), 0, s, a); \
    } else {                                                                                           \
      hipLaunchKernelGGL((k_bp_attn<WT, D, GG, GG, 4>), grid, dim3(64 * kQT), 0, s, a);                \
    }                                                                                                  \
    break;
    EE_ATTN_G(1) EE_ATTN_G(2) EE_ATTN_G(3) EE_ATTN_G(4) EE_ATTN_G(5) EE_ATTN_G(6) EE_ATTN_G(7) EE_ATTN_G(8)
#undef EE_ATTN_G
    default: return hipErrorInvalidValue;
  }
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
  // tiles of 64 x 64 (more than 16 positions) and 16 x 64 (at most 16); on
  // the matrix cores 128 rows x 64 positions and, for at most 16 positions,
  // 32 rows (two row blocks) x 16
  const size_t a = static_cast<size_t>((N_max + 63) / 64) * ((max_positions + 63) / 64);
  const size_t b = static_cast<size_t>((N_max + 31) / 32);
  return std::max(a, b);
}

}  // namespace ee
