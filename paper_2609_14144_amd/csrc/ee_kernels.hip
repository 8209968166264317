// HIP kernels of the gated early-exit decode step for gfx950 (CDNA4).
//
// Every operation of the step is a "phase": a device function that processes
// work items wg, wg + nwg, ... of one operation. The same phases run either
// as one kernel per operation (blockIdx.x = wg) or inside one persistent
// cooperative kernel that runs whole decode steps, separated by grid barriers,
// with the exit branch taken on the device.
//
// Numerics: weights bf16 (or fp32), activations and accumulation fp32, KV
// cache entries stored in the weight type (round to nearest even for bf16).
// Batch-1 decode is bound by HBM bandwidth: each weight byte is read once per
// step with 16-byte coalesced loads; activations stay in LDS.
//
// Cross-workgroup communication (MI355X has one L2 per XCD; the L2s are not
// coherent with each other for ordinary accesses):
//   * every value another workgroup reads later in the same launch
//     (activations, partial results, the step record, KV entries) is written
//     with device-coherent stores (relaxed agent-scope atomic stores, which
//     write through the XCD's L2);
//   * activations, partial results and the step record are read with
//     device-coherent loads;
//   * weights are read-only; KV cache rows are read with plain loads: a KV
//     row is written once (at its position's step) before any workgroup reads
//     it in that launch, and every row starts on a 128-byte line of its own,
//     so no L2 can hold a stale copy;
//   * a producer waits for its own stores to complete (s_waitcnt vmcnt(0))
//     before signalling with one relaxed atomic. No L2 writeback or
//     invalidate is ever issued.
#include <math.h>
#include <stdint.h>

#include "ee_internal.h"

namespace ee {

// ---------------------------------------------------------------------------
// coherent accesses
// ---------------------------------------------------------------------------
__device__ __forceinline__ float ld_coh(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_coh(const int* p) {
  return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh_u32(void* p, uint32_t v) {
  __hip_atomic_store(static_cast<uint32_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh_u64(void* p, uint64_t v) {
  __hip_atomic_store(static_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh2(float* p, float a, float b) {  // p 8-byte aligned
  st_coh_u64(p, static_cast<uint64_t>(__float_as_uint(a)) |
                    (static_cast<uint64_t>(__float_as_uint(b)) << 32));
}
// Wait until this wave's outstanding memory operations have completed; also a
// compiler barrier for memory accesses.
__device__ __forceinline__ void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// ---------------------------------------------------------------------------
// storage types
// ---------------------------------------------------------------------------
template <typename WT>
struct Elem;

template <>
struct Elem<uint16_t> {  // bf16 bit patterns
  static constexpr int N = 8;  // elements per 16-byte chunk
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
  __device__ static inline float load(const uint16_t* p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
  }
  __device__ static inline uint32_t bits(float x) {  // round to nearest even
    uint32_t u = __float_as_uint(x);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
  }
  // two adjacent elements with one coherent store
  __device__ static inline void store_pair(uint16_t* p, float a, float b) {
    st_coh_u32(p, bits(a) | (bits(b) << 16));
  }
};

template <>
struct Elem<float> {
  static constexpr int N = 4;
  __device__ static inline void unpack(const uint4& w, float* f) {
    f[0] = __uint_as_float(w.x);
    f[1] = __uint_as_float(w.y);
    f[2] = __uint_as_float(w.z);
    f[3] = __uint_as_float(w.w);
  }
  __device__ static inline float load(const float* p) { return *p; }
  __device__ static inline void store_pair(float* p, float a, float b) { st_coh2(p, a, b); }
};

// ---------------------------------------------------------------------------
// reductions
// ---------------------------------------------------------------------------
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

template <int R>
__device__ inline void wave_sum_n(float (&v)[R]) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
#pragma unroll
    for (int r = 0; r < R; ++r) v[r] += __shfl_xor(v[r], off, 64);
  }
}

// Sum over the workgroup; every thread gets the total. Fixed order.
__device__ inline float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) s += red[i];
  return s;
}

// xs[i] = x[i] / sqrt(mean(x^2) + eps) * g[i]  (x fp32, written by other workgroups)
__device__ inline void rmsnorm_to_lds(const float* x, const float* __restrict__ g, int n, float eps,
                                      float* xs, float* red) {
  __syncthreads();  // xs may still be read by a previous item
  float ss = 0.f;
  for (int i = threadIdx.x; i < n; i += kWG) {
    const float v = ld_coh(x + i);
    xs[i] = v;
    ss = fmaf(v, v, ss);
  }
  const float r = rsqrtf(block_sum(ss, red) / static_cast<float>(n) + eps);
  for (int i = threadIdx.x; i < n; i += kWG) xs[i] = xs[i] * r * g[i];
  __syncthreads();
}

__device__ inline void copy_to_lds(const float* x, int n, float* xs) {
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += kWG) xs[i] = ld_coh(x + i);
  __syncthreads();
}

// ---------------------------------------------------------------------------
// GEMV core: acc[r] += sum over 16-byte chunks c in [c0 + lane, c1) step 64 of
// W[row r][chunk c] . xs[chunk c]. Rows beyond nvalid re-read the last valid
// row (results discarded by the caller), so no access leaves the matrix.
// ---------------------------------------------------------------------------
template <int N>
__device__ inline void load_x(const float* xs, int c, float* x) {
  const float4* p = reinterpret_cast<const float4*>(xs + c * N);
  const float4 a = p[0];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  if constexpr (N == 8) {
    const float4 b = p[1];
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
}

template <typename WT>
__device__ inline float fma_chunk(const uint4& w, const float* x, float acc) {
  constexpr int N = Elem<WT>::N;
  float f[N];
  Elem<WT>::unpack(w, f);
#pragma unroll
  for (int e = 0; e < N; ++e) acc = fmaf(f[e], x[e], acc);
  return acc;
}

template <typename WT, int R>
__device__ inline void rows_dot(const WT* __restrict__ W, int64_t ld, int nvalid,
                                const float* __restrict__ xs, int c0, int c1, int lane,
                                float (&acc)[R]) {
  constexpr int N = Elem<WT>::N;
  const uint4* wr[R];
#pragma unroll
  for (int r = 0; r < R; ++r)
    wr[r] = reinterpret_cast<const uint4*>(W + static_cast<int64_t>(r < nvalid ? r : nvalid - 1) * ld);
  int c = c0 + lane;
  for (; c + 64 < c1; c += 128) {
    uint4 w0[R], w1[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      w0[r] = wr[r][c];
      w1[r] = wr[r][c + 64];
    }
    float x0[N], x1[N];
    load_x<N>(xs, c, x0);
    load_x<N>(xs, c + 64, x1);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      acc[r] = fma_chunk<WT>(w0[r], x0, acc[r]);
      acc[r] = fma_chunk<WT>(w1[r], x1, acc[r]);
    }
  }
  if (c < c1) {
    uint4 w0[R];
#pragma unroll
    for (int r = 0; r < R; ++r) w0[r] = wr[r][c];
    float x0[N];
    load_x<N>(xs, c, x0);
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = fma_chunk<WT>(w0[r], x0, acc[r]);
  }
}

// ---------------------------------------------------------------------------
// KV cache: pool[layer][page][kv_head][slot][D]. Key rows are stored with the
// rotate-half pairs interleaved (element 2i = dimension i, element 2i+1 =
// dimension i + D/2), query vectors use the same order, so q.k is unchanged;
// value rows are in natural order.
// ---------------------------------------------------------------------------
__device__ inline int64_t kv_offset(const DevParams& p, int l, int pos, int kvh) {
  const int page = p.block_table[pos >> p.page_shift];
  const int slot = pos & (p.page_size - 1);
  return static_cast<int64_t>(l) * p.layer_stride +
         ((static_cast<int64_t>(page) * p.K + kvh) * p.page_size + slot) * p.D;
}

// Store the two outputs of row pair (r0, r0+1) of the repacked wqkv matrix:
// q/k pairs are RoPE halves (i, i + D/2), rotated at position pos; v rows are
// consecutive elements.
template <typename WT>
__device__ inline void store_qkv_pair(const DevParams& p, int l, int pos, int r0, float x1, float x2) {
  const int AD = p.A * p.D, KD = p.K * p.D;
  if (r0 < AD + KD) {
    const int head = r0 / p.D;
    const int rl = r0 - head * p.D;  // = 2i
    const int half = p.D >> 1;
    const float c = p.rope_cos[static_cast<int64_t>(pos) * half + (rl >> 1)];
    const float s = p.rope_sin[static_cast<int64_t>(pos) * half + (rl >> 1)];
    const float y1 = x1 * c - x2 * s;
    const float y2 = x2 * c + x1 * s;
    if (r0 < AD) {
      st_coh2(p.q + r0, y1, y2);
    } else {
      WT* kp = static_cast<WT*>(p.kpool) + kv_offset(p, l, pos, head - p.A) + rl;
      Elem<WT>::store_pair(kp, y1, y2);
    }
  } else {
    const int j = r0 - AD - KD;
    const int kvh = j / p.D, d = j - kvh * p.D;
    WT* vp = static_cast<WT*>(p.vpool) + kv_offset(p, l, pos, kvh) + d;
    Elem<WT>::store_pair(vp, x1, x2);
  }
}

__device__ inline int step_token(const DevParams& p, int step) {
  int tok = p.force_tok ? p.force_tok[step] : ld_coh(&p.ctl->next_token);
  if (tok < 0 || tok >= p.V) {
    if (threadIdx.x == 0) atomicMax(&p.ctl->error, kErrToken);
    tok = 0;
  }
  return tok;
}

// ---------------------------------------------------------------------------
// phase: RMSNorm + QKV projection + RoPE + KV append (one layer)
// For layer 0 the input is the embedding row of the step's token, and
// workgroup 0 also initialises the residual stream h with it.
// ---------------------------------------------------------------------------
template <typename WT>
__device__ void phase_qkv(const DevParams& p, int l, int pos, int step, int wg, int nwg, float* xs,
                          float* red) {
  const int pairs = p.qkv_rows >> 1;
  const int items = (pairs + kWaves - 1) / kWaves;
  if (wg >= items) return;
  const LayerW lw = p.layers[l];
  if (l == 0) {
    const int tok = step_token(p, step);
    const WT* e = static_cast<const WT*>(p.embed) + static_cast<int64_t>(tok) * p.H;
    __syncthreads();
    float ss = 0.f;
    for (int i = threadIdx.x; i < p.H; i += kWG) {
      const float v = Elem<WT>::load(e + i);
      xs[i] = v;
      ss = fmaf(v, v, ss);
      if (wg == 0) st_coh(p.h + i, v);
    }
    const float r = rsqrtf(block_sum(ss, red) / static_cast<float>(p.H) + p.eps);
    for (int i = threadIdx.x; i < p.H; i += kWG) xs[i] = xs[i] * r * lw.g_attn[i];
    __syncthreads();
    if (wg == 0 && threadIdx.x == 0) st_coh(&p.ctl->exited, 0);
  } else {
    rmsnorm_to_lds(p.h, lw.g_attn, p.H, p.eps, xs, red);
  }
  const WT* W = static_cast<const WT*>(lw.wqkv);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = p.H / Elem<WT>::N;
  for (int it = wg; it < items; it += nwg) {
    const int pair = it * kWaves + wave;
    if (pair >= pairs) continue;
    const int r0 = 2 * pair;
    float acc[2] = {0.f, 0.f};
    rows_dot<WT, 2>(W + static_cast<int64_t>(r0) * p.H, p.H, 2, xs, 0, nch, lane, acc);
    wave_sum_n<2>(acc);
    if (lane == 0) store_qkv_pair<WT>(p, l, pos, r0, acc[0], acc[1]);
  }
}

// ---------------------------------------------------------------------------
// phase: decode attention over positions 0..pos, grouped-query. A wave item
// is (kv head, split of kAttnSplit = 64 positions). Scores: lanes own
// positions (q of the G query heads sharing the kv head broadcast from LDS).
// Weighted V: groups of D/N lanes own one position's row in 16-byte chunks.
// Each item writes a partial (max, sum of exp, weighted V); the last item of a
// kv head to finish merges the splits in index order into o.
// ---------------------------------------------------------------------------
__host__ __device__ inline int attn_lds_floats(int G, int D) {
  return kWaves * (G * D + G * kAttnSplit + 2 * kAttnSplit);
}

template <typename WT>
__device__ void phase_attn(const DevParams& p, int l, int pos, int wg, int nwg, float* lds) {
  constexpr int N = Elem<WT>::N;
  const int T = pos + 1;
  const int nsplit = (T + kAttnSplit - 1) / kAttnSplit;
  const int items = p.K * nsplit;
  const int witems = (items + kWaves - 1) / kWaves;
  if (wg >= witems) return;
  const int G = p.G, D = p.D;
  const int PS = D + 2;  // partial record: m, l, acc[D]
  const int LPP = D / N, PPW = 64 / LPP;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int sub = lane / LPP, dl = lane - sub * LPP;
  float* qw = lds + wave * (G * D + G * kAttnSplit + 2 * kAttnSplit);  // [G][D] scaled q
  float* pw = qw + G * D;                                              // [G][64] exp(s - m)
  int64_t* offw = reinterpret_cast<int64_t*>(pw + G * kAttnSplit);     // [64] row offsets
  const WT* kp = static_cast<const WT*>(p.kpool);
  const WT* vp = static_cast<const WT*>(p.vpool);

  for (int wit = wg; wit < witems; wit += nwg) {
    const int item = wit * kWaves + wave;
    const bool active = item < items;
    const int kvh = active ? item / nsplit : 0;
    const int sp = active ? item - kvh * nsplit : 0;
    const int s0 = sp * kAttnSplit;
    const int ns = active ? min(kAttnSplit, T - s0) : 0;
    __syncthreads();  // the previous item's LDS reads are done
    if (active) {
      for (int i = lane; i < G * D; i += 64) qw[i] = ld_coh(p.q + kvh * G * D + i) * p.attn_scale;
      offw[lane] = lane < ns ? kv_offset(p, l, s0 + lane, kvh) : 0;
    }
    __syncthreads();
    const bool valid = lane < ns;
    float sc[kMaxGroup];
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) sc[g] = 0.f;
    if (valid) {
      const uint4* kr = reinterpret_cast<const uint4*>(kp + offw[lane]);
#pragma unroll 4
      for (int c = 0; c < D / N; ++c) {
        float kf[N];
        Elem<WT>::unpack(kr[c], kf);
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) {
          if (g < G) {
            const float* qg = qw + g * D + c * N;
#pragma unroll
            for (int e = 0; e < N; ++e) sc[g] = fmaf(qg[e], kf[e], sc[g]);
          }
        }
      }
    }
    float mg[kMaxGroup], lg[kMaxGroup];
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) {
      mg[g] = 0.f;
      lg[g] = 0.f;
      if (g < G) {
        const float v = valid ? sc[g] : -INFINITY;
        const float m = wave_max(v);
        const float e = valid ? expf(v - m) : 0.f;
        mg[g] = m;
        lg[g] = wave_sum(e);
        if (active) pw[g * kAttnSplit + lane] = e;
      }
    }
    __syncthreads();
    if (!active) continue;
    // weighted V: lanes (sub, dl) take position j0 + sub, dimensions dl*N .. dl*N + N
    float acc[kMaxGroup][N];
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g)
#pragma unroll
      for (int e = 0; e < N; ++e) acc[g][e] = 0.f;
#pragma unroll 2
    for (int j0 = 0; j0 < ns; j0 += PPW) {
      const int j = j0 + sub;
      if (j < ns) {
        const uint4 vw = *reinterpret_cast<const uint4*>(vp + offw[j] + dl * N);
        float vf[N];
        Elem<WT>::unpack(vw, vf);
#pragma unroll
        for (int g = 0; g < kMaxGroup; ++g) {
          if (g < G) {
            const float pj = pw[g * kAttnSplit + j];
#pragma unroll
            for (int e = 0; e < N; ++e) acc[g][e] = fmaf(pj, vf[e], acc[g][e]);
          }
        }
      }
    }
    for (int off = LPP; off < 64; off <<= 1) {
#pragma unroll
      for (int g = 0; g < kMaxGroup; ++g)
        if (g < G)
#pragma unroll
          for (int e = 0; e < N; ++e) acc[g][e] += __shfl_xor(acc[g][e], off, 64);
    }
    float* part = p.attn_part + (static_cast<int64_t>(kvh) * p.max_splits + sp) * G * PS;
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) {
      if (g < G) {
        if (sub == 0) {
#pragma unroll
          for (int e = 0; e < N; e += 2)
            st_coh2(part + g * PS + 2 + dl * N + e, acc[g][e], acc[g][e + 1]);
        }
        if (lane == 0) st_coh2(part + g * PS, mg[g], lg[g]);
      }
    }
    // the last item of this kv head to finish merges all splits into o
    wait_stores();
    uint32_t old = 0;
    if (lane == 0)
      old = __hip_atomic_fetch_add(&p.counters->attn[kvh * 64], 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    old = __shfl(old, 0, 64);
    if (old == static_cast<uint32_t>(nsplit - 1)) {
      const float* base = p.attn_part + static_cast<int64_t>(kvh) * p.max_splits * G * PS;
      for (int idx = lane; idx < G * D; idx += 64) {
        const int g = idx / D, d = idx - g * D;
        float M = -INFINITY;
        for (int s2 = 0; s2 < nsplit; ++s2) M = fmaxf(M, ld_coh(base + (s2 * G + g) * PS));
        float den = 0.f, num = 0.f;
        for (int s2 = 0; s2 < nsplit; ++s2) {
          const float* rec = base + (s2 * G + g) * PS;
          const float wgt = expf(ld_coh(rec) - M);
          den = fmaf(wgt, ld_coh(rec + 1), den);
          num = fmaf(wgt, ld_coh(rec + 2 + d), num);
        }
        st_coh(p.o + (kvh * G + g) * D + d, num / den);
      }
      if (lane == 0)
        __hip_atomic_store(&p.counters->attn[kvh * 64], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// ---------------------------------------------------------------------------
// phase: out[r] (+)= W[r] . x for rows of a [rows][cols] matrix, x staged in
// LDS. Items of kWaves * R rows, one R-row group per wave.
// mode 0: out = acc + bias (bias may be null); mode 1: out += acc.
// ---------------------------------------------------------------------------
template <typename WT, int R>
__device__ void phase_gemv(const WT* __restrict__ W, int rows, int cols, const float* x, float* out,
                           const float* bias, int mode, int wg, int nwg, float* xs) {
  const int items = (rows + kWaves * R - 1) / (kWaves * R);
  if (wg >= items) return;
  copy_to_lds(x, cols, xs);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = cols / Elem<WT>::N;
  for (int it = wg; it < items; it += nwg) {
    const int r0 = (it * kWaves + wave) * R;
    if (r0 >= rows) continue;
    const int nv = min(R, rows - r0);
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
    rows_dot<WT, R>(W + static_cast<int64_t>(r0) * cols, cols, nv, xs, 0, nch, lane, acc);
    wave_sum_n<R>(acc);
    if (lane == 0) {
      for (int r = 0; r < nv; ++r) {
        const float prev = mode == 1 ? ld_coh(out + r0 + r) : (bias ? bias[r0 + r] : 0.f);
        st_coh(out + r0 + r, prev + acc[r]);
      }
    }
  }
}

// Same with the K dimension split over the workgroup's waves: item = R rows,
// wave w handles chunk range w of kWaves; partial sums meet in LDS. out += acc.
template <typename WT, int R>
__device__ void phase_gemv_splitk(const WT* __restrict__ W, int rows, int cols, const float* x,
                                  float* out, int wg, int nwg, float* xs, float* red) {
  const int items = (rows + R - 1) / R;
  if (wg >= items) return;
  copy_to_lds(x, cols, xs);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = cols / Elem<WT>::N;
  const int cb = nch * wave / kWaves, ce = nch * (wave + 1) / kWaves;
  for (int it = wg; it < items; it += nwg) {
    const int r0 = it * R;
    const int nv = min(R, rows - r0);
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
    rows_dot<WT, R>(W + static_cast<int64_t>(r0) * cols, cols, nv, xs, cb, ce, lane, acc);
    wave_sum_n<R>(acc);
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < R; ++r) red[wave * R + r] = acc[r];
    }
    __syncthreads();
    if (threadIdx.x < nv) {
      float s = 0.f;
      for (int w = 0; w < kWaves; ++w) s += red[w * R + threadIdx.x];
      st_coh(out + r0 + threadIdx.x, ld_coh(out + r0 + threadIdx.x) + s);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// phase: RMSNorm + gate/up projection + SiLU(gate) * up. Interleaved rows.
// ---------------------------------------------------------------------------
__device__ inline float silu(float x) { return x / (1.f + expf(-x)); }

template <typename WT>
__device__ void phase_gateup(const DevParams& p, int l, int wg, int nwg, float* xs, float* red) {
  const int items = (p.F + 2 * kWaves - 1) / (2 * kWaves);
  if (wg >= items) return;
  const LayerW lw = p.layers[l];
  rmsnorm_to_lds(p.h, lw.g_mlp, p.H, p.eps, xs, red);
  const WT* W = static_cast<const WT*>(lw.wgu);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = p.H / Elem<WT>::N;
  for (int it = wg; it < items; it += nwg) {
    const int j0 = (it * kWaves + wave) * 2;
    if (j0 >= p.F) continue;
    const int nv = min(4, 2 * (p.F - j0));
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    rows_dot<WT, 4>(W + static_cast<int64_t>(2 * j0) * p.H, p.H, nv, xs, 0, nch, lane, acc);
    wave_sum_n<4>(acc);
    if (lane == 0) {
      if (nv == 4) st_coh2(p.a + j0, silu(acc[0]) * acc[1], silu(acc[2]) * acc[3]);
      else st_coh(p.a + j0, silu(acc[0]) * acc[1]);
    }
  }
}

// ---------------------------------------------------------------------------
// phase: head = RMSNorm(src; g_final) -> unembedding -> online (max, argmax,
// sum exp, second max) over the vocabulary, never writing logits (unless a
// debug buffer is given). Each workgroup owns a contiguous row range and
// writes one partial; the last workgroup merges the partials with a fixed
// tree, takes the gate decision (readout) or the final token, and emits.
// ---------------------------------------------------------------------------
struct Stat {
  float m;    // max logit
  float s;    // sum of exp(logit - m)
  float m2;   // second largest logit (equal to m on ties)
  int idx;    // argmax, lowest index among ties
};

__device__ inline Stat stat_empty() { return Stat{-INFINITY, 0.f, -INFINITY, 0x7fffffff}; }

__device__ inline void stat_push(Stat& st, float v, int r) {
  if (v > st.m) {
    st.s = st.s * expf(st.m - v) + 1.f;
    st.m2 = st.m;
    st.m = v;
    st.idx = r;
  } else {
    st.s += expf(v - st.m);
    st.m2 = fmaxf(st.m2, v);
  }
}

__device__ inline Stat stat_merge(Stat a, Stat b) {
  if (b.s == 0.f) return a;
  if (a.s == 0.f) return b;
  const bool bw = b.m > a.m || (b.m == a.m && b.idx < a.idx);
  Stat w = bw ? b : a;
  const Stat o = bw ? a : b;
  w.s = w.s + o.s * expf(o.m - w.m);
  w.m2 = fmaxf(w.m2, o.m);
  return w;
}

template <typename WT>
__device__ void phase_head(const DevParams& p, int readout, int step, int wg, int nwg, float* xs,
                           float* red, float* stl) {
  rmsnorm_to_lds(readout ? p.z : p.h, p.g_final, p.H, p.eps, xs, red);
  const WT* E = static_cast<const WT*>(p.embed);
  float* dbg = readout ? p.dbg_logits_r : p.dbg_logits_f;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = p.H / Elem<WT>::N;
  const int rb = static_cast<int>(static_cast<int64_t>(p.V) * wg / nwg);
  const int re = static_cast<int>(static_cast<int64_t>(p.V) * (wg + 1) / nwg);
  constexpr int R = 4;
  Stat st = stat_empty();
  for (int r0 = rb + wave * R; r0 < re; r0 += kWaves * R) {
    const int nv = min(R, re - r0);
    float acc[R] = {0.f, 0.f, 0.f, 0.f};
    rows_dot<WT, R>(E + static_cast<int64_t>(r0) * p.H, p.H, nv, xs, 0, nch, lane, acc);
    wave_sum_n<R>(acc);
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (r < nv) stat_push(st, acc[r], r0 + r);
    if (dbg && lane == 0)
      for (int r = 0; r < nv; ++r) dbg[r0 + r] = acc[r];
  }
  __shared__ int last_flag;
  __syncthreads();
  if (lane == 0) {
    stl[wave * 4 + 0] = st.m;
    stl[wave * 4 + 1] = st.s;
    stl[wave * 4 + 2] = st.m2;
    stl[wave * 4 + 3] = __int_as_float(st.idx);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    Stat t = stat_empty();
    for (int w = 0; w < kWaves; ++w)
      t = stat_merge(t, Stat{stl[w * 4], stl[w * 4 + 1], stl[w * 4 + 2], __float_as_int(stl[w * 4 + 3])});
    float* part = p.head_part + static_cast<int64_t>(wg) * 4;
    st_coh2(part, t.m, t.s);
    st_coh2(part + 2, t.m2, __int_as_float(t.idx));
    wait_stores();
    const uint32_t old = __hip_atomic_fetch_add(&p.counters->head[0], 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    last_flag = (old == static_cast<uint32_t>(nwg - 1));
  }
  __syncthreads();
  if (!last_flag) return;
  Stat t = stat_empty();
  for (int i = threadIdx.x; i < nwg; i += kWG) {
    const float* part = p.head_part + static_cast<int64_t>(i) * 4;
    t = stat_merge(t, Stat{ld_coh(part), ld_coh(part + 1), ld_coh(part + 2),
                           __float_as_int(ld_coh(part + 3))});
  }
  stl[threadIdx.x * 4 + 0] = t.m;
  stl[threadIdx.x * 4 + 1] = t.s;
  stl[threadIdx.x * 4 + 2] = t.m2;
  stl[threadIdx.x * 4 + 3] = __int_as_float(t.idx);
  __syncthreads();
  for (int stride = kWG / 2; stride > 0; stride >>= 1) {
    if (threadIdx.x < stride) {
      const float* a = stl + threadIdx.x * 4;
      const float* b = stl + (threadIdx.x + stride) * 4;
      const Stat r = stat_merge(Stat{a[0], a[1], a[2], __float_as_int(a[3])},
                                Stat{b[0], b[1], b[2], __float_as_int(b[3])});
      float* d = stl + threadIdx.x * 4;
      d[0] = r.m;
      d[1] = r.s;
      d[2] = r.m2;
      d[3] = __int_as_float(r.idx);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int idx = __float_as_int(stl[3]);
    const float conf = 1.f / stl[1];
    StepCtl* c = p.ctl;
    __hip_atomic_store(&p.counters->head[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (readout) {
      const int would = conf > p.tau;
      const int fe = p.force_exit ? p.force_exit[step] : -1;
      const int ex = fe < 0 ? would : fe;
      st_coh(&c->readout_token, idx);
      st_coh(&c->conf, conf);
      st_coh(&c->would_exit, would);
      st_coh(&c->exited, ex);
      if (ex) {
        st_coh(&c->next_token, idx);
        if (p.ring_tok) {
          p.ring_tok[step] = idx;
          p.ring_exit[step] = 1;
          p.ring_conf[step] = conf;
          p.ring_would[step] = would;
        }
      }
    } else {
      const int gated = p.exit_layer > 0;
      st_coh(&c->full_token, idx);
      st_coh(&c->conf_full, conf);
      st_coh(&c->next_token, idx);
      if (p.ring_tok) {
        p.ring_tok[step] = idx;
        p.ring_exit[step] = 0;
        p.ring_conf[step] = gated ? ld_coh(&c->conf) : conf;
        p.ring_would[step] = gated ? ld_coh(&c->would_exit) : 0;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// phase: KV-absence fill after an exit. For every skipped layer l (exit_layer
// .. L-1, 0-based): a = RMSNorm(h_exit; g_attn[l]); K_l[pos] = RoPE(W_k,l a),
// V_l[pos] = W_v,l a. Items are layer-major groups of kWaves row pairs.
// ---------------------------------------------------------------------------
template <typename WT>
__device__ void phase_fill(const DevParams& p, int pos, int wg, int nwg, float* xs, float* red) {
  const int nl = p.L - p.exit_layer;
  const int KD = p.K * p.D;                 // row pairs per layer (k and v rows: 2*KD)
  const int ipl = (KD + kWaves - 1) / kWaves;
  const int items = nl * ipl;
  if (wg >= items) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = p.H / Elem<WT>::N;
  const int AD = p.A * p.D;
  int cur = -1;
  for (int it = wg; it < items; it += nwg) {
    const int l = p.exit_layer + it / ipl;
    const LayerW lw = p.layers[l];
    if (l != cur) {
      rmsnorm_to_lds(p.h_exit, lw.g_attn, p.H, p.eps, xs, red);
      cur = l;
    }
    const int pair = (it % ipl) * kWaves + wave;
    if (pair >= KD) continue;
    const int r0 = AD + 2 * pair;
    float acc[2] = {0.f, 0.f};
    rows_dot<WT, 2>(static_cast<const WT*>(lw.wqkv) + static_cast<int64_t>(r0) * p.H, p.H, 2, xs, 0,
                    nch, lane, acc);
    wave_sum_n<2>(acc);
    if (lane == 0) store_qkv_pair<WT>(p, l, pos, r0, acc[0], acc[1]);
  }
}

// readout: z = W_r h + b_r; workgroup 0 also keeps h as h_exit.
template <typename WT>
__device__ void phase_readout(const DevParams& p, int wg, int nwg, float* xs) {
  if (wg == 0)
    for (int i = threadIdx.x; i < p.H; i += kWG) st_coh(p.h_exit + i, ld_coh(p.h + i));
  phase_gemv<WT, 2>(static_cast<const WT*>(p.ro_w), p.H, p.H, p.h, p.z, p.ro_b, 0, wg, nwg, xs);
}

// ---------------------------------------------------------------------------
// LDS layout: xs [vec] | red [64] | stat [kWG * 4]
// ---------------------------------------------------------------------------
__host__ __device__ inline int lds_vec_floats(const DevParams& p) {
  int v = p.H;
  if (p.F > v) v = p.F;
  if (p.A * p.D > v) v = p.A * p.D;
  const int am = attn_lds_floats(p.G, p.D);
  if (am > v) v = am;
  return (v + 63) & ~63;
}

size_t lds_bytes(const DevParams& p) {
  return static_cast<size_t>(lds_vec_floats(p) + 64 + kWG * 4) * sizeof(float);
}

struct Lds {
  float* xs;
  float* red;
  float* stl;
};

__device__ inline Lds lds_carve(const DevParams& p, float* smem) {
  const int v = lds_vec_floats(p);
  return Lds{smem, smem + v, smem + v + 64};
}

// ---------------------------------------------------------------------------
// one-kernel-per-operation drivers
// ---------------------------------------------------------------------------
enum OpKind : int {
  kOpQkv = 0, kOpAttn, kOpWo, kOpGateUp, kOpDown, kOpReadout, kOpHeadR, kOpHeadF, kOpFill
};

template <typename WT, int OP>
__global__ __launch_bounds__(kWG) void k_op(DevParams p, int l, int pos, int step, int skip_if_exited) {
  extern __shared__ float smem[];
  if (skip_if_exited && ld_coh(&p.ctl->exited)) return;
  const Lds s = lds_carve(p, smem);
  const int wg = blockIdx.x, nwg = gridDim.x;
  if constexpr (OP == kOpQkv) phase_qkv<WT>(p, l, pos, step, wg, nwg, s.xs, s.red);
  if constexpr (OP == kOpAttn) phase_attn<WT>(p, l, pos, wg, nwg, s.xs);
  if constexpr (OP == kOpWo)
    phase_gemv<WT, 2>(static_cast<const WT*>(p.layers[l].wo), p.H, p.A * p.D, p.o, p.h, nullptr, 1, wg,
                      nwg, s.xs);
  if constexpr (OP == kOpGateUp) phase_gateup<WT>(p, l, wg, nwg, s.xs, s.red);
  if constexpr (OP == kOpDown)
    phase_gemv_splitk<WT, 2>(static_cast<const WT*>(p.layers[l].wd), p.H, p.F, p.a, p.h, wg, nwg, s.xs,
                             s.red);
  if constexpr (OP == kOpReadout) phase_readout<WT>(p, wg, nwg, s.xs);
  if constexpr (OP == kOpHeadR) phase_head<WT>(p, 1, step, wg, nwg, s.xs, s.red, s.stl);
  if constexpr (OP == kOpHeadF) phase_head<WT>(p, 0, step, wg, nwg, s.xs, s.red, s.stl);
  if constexpr (OP == kOpFill)
    if (ld_coh(&p.ctl->exited)) phase_fill<WT>(p, pos, wg, nwg, s.xs, s.red);
}

static int op_grid(const DevParams& p, int op, int pos, int head_wgs) {
  switch (op) {
    case kOpQkv: return ((p.qkv_rows >> 1) + kWaves - 1) / kWaves;
    case kOpAttn: return (p.K * ((pos + 1 + kAttnSplit - 1) / kAttnSplit) + kWaves - 1) / kWaves;
    case kOpWo: return (p.H + kWaves * 2 - 1) / (kWaves * 2);
    case kOpGateUp: return (p.F + 2 * kWaves - 1) / (2 * kWaves);
    case kOpDown: return (p.H + 1) / 2;
    case kOpReadout: return (p.H + kWaves * 2 - 1) / (kWaves * 2);
    case kOpHeadR:
    case kOpHeadF: return head_wgs;
    case kOpFill: {
      const int nl = p.L - p.exit_layer;
      const int ipl = (p.K * p.D + kWaves - 1) / kWaves;
      return nl * ipl > 0 ? nl * ipl : 1;
    }
  }
  return 1;
}

template <typename WT>
static hipError_t op(const DevParams& p, int kind, int l, int pos, int step, int skip, int head_wgs,
                     hipStream_t s) {
  const int grid = op_grid(p, kind, pos, head_wgs);
  const size_t lds = lds_bytes(p);
  switch (kind) {
#define EE_OP_CASE(K)                                                                        \
  case K:                                                                                    \
    hipLaunchKernelGGL((k_op<WT, K>), dim3(grid), dim3(kWG), lds, s, p, l, pos, step, skip); \
    break;
    EE_OP_CASE(kOpQkv)
    EE_OP_CASE(kOpAttn)
    EE_OP_CASE(kOpWo)
    EE_OP_CASE(kOpGateUp)
    EE_OP_CASE(kOpDown)
    EE_OP_CASE(kOpReadout)
    EE_OP_CASE(kOpHeadR)
    EE_OP_CASE(kOpHeadF)
    EE_OP_CASE(kOpFill)
#undef EE_OP_CASE
  }
  return hipGetLastError();
}

template <typename WT>
static hipError_t layer_ops(const DevParams& p, int l, int pos, int step, int skip, int hw,
                            hipStream_t s) {
  hipError_t e;
  if ((e = op<WT>(p, kOpQkv, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  if ((e = op<WT>(p, kOpAttn, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  if ((e = op<WT>(p, kOpWo, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  if ((e = op<WT>(p, kOpGateUp, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  return op<WT>(p, kOpDown, l, pos, step, skip, hw, s);
}

// One decode step (or one prompt position when emit_head == 0) per op.
template <typename WT>
static hipError_t step_per_op(const DevParams& p, int pos, int step, int emit_head, int hw,
                              hipStream_t s) {
  hipError_t e;
  const int Le = p.exit_layer;
  for (int l = 0; l < Le; ++l)
    if ((e = layer_ops<WT>(p, l, pos, step, 0, hw, s)) != hipSuccess) return e;
  if (Le > 0) {
    if ((e = op<WT>(p, kOpReadout, 0, pos, step, 0, hw, s)) != hipSuccess) return e;
    if ((e = op<WT>(p, kOpHeadR, 0, pos, step, 0, hw, s)) != hipSuccess) return e;
    if ((e = op<WT>(p, kOpFill, 0, pos, step, 0, hw, s)) != hipSuccess) return e;
  }
  for (int l = Le; l < p.L; ++l)
    if ((e = layer_ops<WT>(p, l, pos, step, Le > 0, hw, s)) != hipSuccess) return e;
  if (emit_head) return op<WT>(p, kOpHeadF, 0, pos, step, Le > 0, hw, s);
  return hipSuccess;
}

hipError_t launch_decode_per_op(const DevParams& p, int wbf16, int pos0, int n, int head_wgs,
                                hipStream_t s) {
  for (int i = 0; i < n; ++i) {
    const hipError_t e = wbf16 ? step_per_op<uint16_t>(p, pos0 + i, i, 1, head_wgs, s)
                               : step_per_op<float>(p, pos0 + i, i, 1, head_wgs, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_prefill_per_op(const DevParams& p, int wbf16, int pos0, const int32_t* d_tokens,
                                 int n, int head_wgs, hipStream_t s) {
  DevParams q = p;
  q.exit_layer = 0;
  q.force_tok = d_tokens;
  q.force_exit = nullptr;
  for (int i = 0; i < n; ++i) {
    const int emit = (i == n - 1);
    const hipError_t e = wbf16 ? step_per_op<uint16_t>(q, pos0 + i, i, emit, head_wgs, s)
                               : step_per_op<float>(q, pos0 + i, i, emit, head_wgs, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

__global__ __launch_bounds__(kWG) void k_copy_vec(float* dst, const float* src, int n) {
  for (int i = blockIdx.x * kWG + threadIdx.x; i < n; i += gridDim.x * kWG) dst[i] = src[i];
}

hipError_t launch_head_eval(const DevParams& p, int wbf16, const float* d_x, int readout, int head_wgs,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_copy_vec, dim3(8), dim3(kWG), 0, s, p.h, d_x, p.H);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (readout) {
    e = wbf16 ? op<uint16_t>(p, kOpReadout, 0, 0, 0, 0, head_wgs, s)
              : op<float>(p, kOpReadout, 0, 0, 0, 0, head_wgs, s);
    if (e != hipSuccess) return e;
  }
  const int kind = readout ? kOpHeadR : kOpHeadF;
  return wbf16 ? op<uint16_t>(p, kind, 0, 0, 0, 0, head_wgs, s)
               : op<float>(p, kind, 0, 0, 0, 0, head_wgs, s);
}

// ---------------------------------------------------------------------------
// persistent cooperative kernel: n whole decode steps in one launch
// ---------------------------------------------------------------------------
constexpr uint64_t kWaitTicks = 400000000ull;  // ~4 s of the 100 MHz wall clock

// All workgroups arrive, then wait for the count to reach target. The wait is
// bounded: on time-out the abort flag is raised and every later wait returns
// at once, so the grid always drains.
__device__ inline void grid_barrier(const DevParams& p, uint32_t& target, int nwg) {
  target += static_cast<uint32_t>(nwg);
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t* ctr = &p.counters->barrier[0];
    __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t t0 = wall_clock64();
    while (true) {
      const uint32_t v = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (static_cast<int32_t>(v - target) >= 0) break;
      if (__hip_atomic_load(&p.ctl->abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
      if (wall_clock64() - t0 > kWaitTicks) {
        __hip_atomic_store(&p.ctl->abort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        atomicMax(&p.ctl->error, kErrBarrier);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
}

template <typename WT>
__device__ void layer_persistent(const DevParams& p, int l, int pos, int step, int wg, int nwg,
                                 const Lds& s, uint32_t& bt) {
  phase_qkv<WT>(p, l, pos, step, wg, nwg, s.xs, s.red);
  grid_barrier(p, bt, nwg);
  phase_attn<WT>(p, l, pos, wg, nwg, s.xs);
  grid_barrier(p, bt, nwg);
  phase_gemv<WT, 2>(static_cast<const WT*>(p.layers[l].wo), p.H, p.A * p.D, p.o, p.h, nullptr, 1, wg,
                    nwg, s.xs);
  grid_barrier(p, bt, nwg);
  phase_gateup<WT>(p, l, wg, nwg, s.xs, s.red);
  grid_barrier(p, bt, nwg);
  phase_gemv_splitk<WT, 2>(static_cast<const WT*>(p.layers[l].wd), p.H, p.F, p.a, p.h, wg, nwg, s.xs,
                           s.red);
  grid_barrier(p, bt, nwg);
}

// prefill != 0: prompt positions, ungated, head only at the last position.
template <typename WT>
__global__ __launch_bounds__(kWG) void k_decode_persistent(DevParams p, int pos0, int n, int prefill) {
  extern __shared__ float smem[];
  const Lds s = lds_carve(p, smem);
  const int wg = blockIdx.x, nwg = gridDim.x;
  uint32_t bt = 0;
  const int Le = p.exit_layer;
  for (int i = 0; i < n; ++i) {
    if (__hip_atomic_load(&p.ctl->abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
    const int pos = pos0 + i;
    for (int l = 0; l < Le; ++l) layer_persistent<WT>(p, l, pos, i, wg, nwg, s, bt);
    int exited = 0;
    if (Le > 0) {
      phase_readout<WT>(p, wg, nwg, s.xs);
      grid_barrier(p, bt, nwg);
      phase_head<WT>(p, 1, i, wg, nwg, s.xs, s.red, s.stl);
      grid_barrier(p, bt, nwg);
      exited = ld_coh(&p.ctl->exited);
    }
    if (exited) {
      phase_fill<WT>(p, pos, wg, nwg, s.xs, s.red);
      grid_barrier(p, bt, nwg);
    } else {
      for (int l = Le; l < p.L; ++l) layer_persistent<WT>(p, l, pos, i, wg, nwg, s, bt);
      if (!prefill || i == n - 1) {
        phase_head<WT>(p, 0, i, wg, nwg, s.xs, s.red, s.stl);
        grid_barrier(p, bt, nwg);
      }
    }
  }
}

__global__ void k_reset_barrier(Counters* c) {
  if (threadIdx.x == 0) c->barrier[0] = 0u;
}

static hipError_t persistent(const DevParams& p, int wbf16, int pos0, int n, int prefill, int nwg,
                             size_t lds, hipStream_t s) {
  hipLaunchKernelGGL(k_reset_barrier, dim3(1), dim3(64), 0, s, p.counters);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  DevParams pp = p;
  void* args[] = {&pp, &pos0, &n, &prefill};
  const void* fn = wbf16 ? reinterpret_cast<const void*>(&k_decode_persistent<uint16_t>)
                         : reinterpret_cast<const void*>(&k_decode_persistent<float>);
  return hipLaunchCooperativeKernel(fn, dim3(nwg), dim3(kWG), args, static_cast<unsigned>(lds), s);
}

hipError_t launch_decode_persistent(const DevParams& p, int wbf16, int pos0, int n, int nwg,
                                    size_t lds, hipStream_t s) {
  return persistent(p, wbf16, pos0, n, 0, nwg, lds, s);
}

hipError_t launch_prefill_persistent(const DevParams& p, int wbf16, int pos0, int n, int nwg,
                                     size_t lds, hipStream_t s) {
  return persistent(p, wbf16, pos0, n, 1, nwg, lds, s);
}

int persistent_max_wgs_per_cu(int wbf16, size_t lds) {
  int nb = 0;
  const void* fn = wbf16 ? reinterpret_cast<const void*>(&k_decode_persistent<uint16_t>)
                         : reinterpret_cast<const void*>(&k_decode_persistent<float>);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, kWG, lds) != hipSuccess) return 0;
  return nb;
}

}  // namespace ee
