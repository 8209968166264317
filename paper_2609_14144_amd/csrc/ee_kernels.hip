// HIP kernels of the gated early-exit decode step for gfx950 (CDNA4).
//
// Every operation of the step is a "phase": a device function that processes
// work items wg, wg + nwg, ... of one operation. The same phases run either
// as one kernel per operation (blockIdx.x = wg) or inside one persistent
// cooperative kernel that runs whole decode steps with the exit branch taken
// on the device. Inside the persistent kernel, phases hand activations to
// each other as tagged words (value + tag of the producing phase): a consumer
// polls its inputs until they carry the expected tag, so consecutive phases
// need no grid barrier; one barrier ends every step and every KV fill.
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
//     before signalling with one relaxed atomic; a tagged word is its own
//     signal (value and tag in one 8-byte store). No L2 writeback or
//     invalidate is ever issued.
//   * a buffer is rewritten only after every reader of its previous contents
//     has produced something the writer itself waited for (the chain
//     q -> o -> h -> a -> h runs through every workgroup that reads), or
//     after a grid barrier (step ends, KV fill).
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

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
  __device__ static inline float round(float x) { return __uint_as_float(bits(x) << 16); }
  // N values that are exactly representable, back into a chunk
  __device__ static inline uint4 pack(const float* f) {
    return make_uint4((__float_as_uint(f[0]) >> 16) | (__float_as_uint(f[1]) & 0xffff0000u),
                      (__float_as_uint(f[2]) >> 16) | (__float_as_uint(f[3]) & 0xffff0000u),
                      (__float_as_uint(f[4]) >> 16) | (__float_as_uint(f[5]) & 0xffff0000u),
                      (__float_as_uint(f[6]) >> 16) | (__float_as_uint(f[7]) & 0xffff0000u));
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
  __device__ static inline float round(float x) { return x; }
  __device__ static inline uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
  }
};

__device__ __forceinline__ uint64_t ld_coh_u64(const void* p) {
  return __hip_atomic_load(static_cast<uint64_t*>(const_cast<void*>(p)), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

constexpr uint64_t kWaitTicks = 400000000ull;  // ~4 s of the 100 MHz wall clock

// ---------------------------------------------------------------------------
// tagged words. Sync describes a phase's inputs and outputs: with poll set
// (persistent kernel), an input word is read until it carries its tag; the
// wait is bounded, and on time-out the abort flag is raised so that every
// later wait returns at once and the grid drains. Without poll (one kernel
// per operation) inputs are complete when the kernel starts.
// ---------------------------------------------------------------------------
struct Sync {
  bool poll;
  uint32_t tin;    // tag of the main input
  uint32_t tres;   // tag of the second input (residual, token, gate record)
  uint32_t tout;   // tag of this phase's outputs
  uint32_t cbase;  // arrivals on this phase's last-arriver counter before it (persistent)
};

__device__ __forceinline__ uint64_t tw_pack(float v, uint32_t tag) {
  return (static_cast<uint64_t>(tag) << 32) | __float_as_uint(v);
}
__device__ __forceinline__ float tw_val(uint64_t w) { return __uint_as_float(static_cast<uint32_t>(w)); }
__device__ __forceinline__ bool tw_ok(uint64_t w, uint32_t tag) { return static_cast<uint32_t>(w >> 32) == tag; }
__device__ __forceinline__ void tw_store(uint64_t* p, float v, uint32_t tag) { st_coh_u64(p, tw_pack(v, tag)); }

__device__ __forceinline__ bool aborted(const DevParams& p) {
  return __hip_atomic_load(&p.ctl->abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
}
__device__ __noinline__ void raise_abort(const DevParams& p, int err) {
  __hip_atomic_store(&p.ctl->abort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  atomicMax(&p.ctl->error, err);
}

// one word, waited for
__device__ inline uint64_t tw_wait(const DevParams& p, const uint64_t* w, uint32_t tag, bool poll) {
  uint64_t v = ld_coh_u64(w);
  if (!poll || tw_ok(v, tag)) return v;
  const uint64_t t0 = wall_clock64();
  while (true) {
    __builtin_amdgcn_s_sleep(2);
    v = ld_coh_u64(w);
    if (tw_ok(v, tag) || aborted(p)) break;
    if (wall_clock64() - t0 > kWaitTicks) {
      raise_abort(p, kErrWait);
      break;
    }
  }
  return v;
}

// Polling loop shared by the readers below: the first pass loads every word;
// later passes (after a short sleep) load again only the words that do not
// carry the tag yet. Without poll, one pass.
#define EE_TW_POLL(KB, ADDR, VALID)                                                 \
  {                                                                               \
    uint64_t t0_ = 0;                                                             \
    for (int pass_ = 0;; ++pass_) {                                               \
      _Pragma("unroll") for (int k = 0; k < (KB); ++k) {                          \
        if ((VALID) && !tw_ok(v[k], tag)) v[k] = ld_coh_u64(ADDR);                \
      }                                                                           \
      if (!poll) break;                                                           \
      bool ready_ = true;                                                         \
      _Pragma("unroll") for (int k = 0; k < (KB); ++k) ready_ = ready_ && tw_ok(v[k], tag); \
      if (ready_ || aborted(p)) break;                                            \
      if (pass_ == 0) t0_ = wall_clock64();                                       \
      else if (wall_clock64() - t0_ > kWaitTicks) {                               \
        raise_abort(p, kErrWait);                                                 \
        break;                                                                    \
      }                                                                           \
      __builtin_amdgcn_s_sleep(2);                                                \
    }                                                                             \
  }

// M words from each of a and b (one lane's own words), waited for together
template <int M>
__device__ inline void tw_read2(const DevParams& p, const uint64_t* a, const uint64_t* b, uint32_t tag,
                                bool poll, float* fa, float* fb) {
  uint64_t v[2 * M];
  const uint64_t none = tw_pack(0.f, tag + 1u);
#pragma unroll
  for (int k = 0; k < 2 * M; ++k) v[k] = none;
  EE_TW_POLL(2 * M, (k < M ? a + k : b + (k - M)), true)
#pragma unroll
  for (int k = 0; k < M; ++k) {
    fa[k] = tw_val(v[k]);
    fb[k] = tw_val(v[M + k]);
  }
}

// n words into xs[0..n) as floats, the whole workgroup; kB words per thread
// are in flight at once. xs is complete after the caller's next barrier.
template <int kB>
__device__ inline void tw_stage(const DevParams& p, const uint64_t* src, int n, uint32_t tag, bool poll,
                                float* xs) {
  const uint64_t none = tw_pack(0.f, tag + 1u);
  for (int base = 0; base < n; base += kB * kWG) {
    uint64_t v[kB];
#pragma unroll
    for (int k = 0; k < kB; ++k) v[k] = base + k * kWG + static_cast<int>(threadIdx.x) < n ? none : tw_pack(0.f, tag);
    EE_TW_POLL(kB, src + base + k * kWG + threadIdx.x, true)
#pragma unroll
    for (int k = 0; k < kB; ++k) {
      const int i = base + k * kWG + static_cast<int>(threadIdx.x);
      if (i < n) xs[i] = tw_val(v[k]);
    }
  }
}

// As tw_stage, for n words src[at(i)] (i < n) gathered into xs[0..n).
template <int kB, typename At>
__device__ inline void tw_gather(const DevParams& p, const uint64_t* src, int n, At at, uint32_t tag, bool poll,
                                 float* xs) {
  const uint64_t none = tw_pack(0.f, tag + 1u);
  for (int base = 0; base < n; base += kB * kWG) {
    uint64_t v[kB];
#pragma unroll
    for (int k = 0; k < kB; ++k) v[k] = base + k * kWG + static_cast<int>(threadIdx.x) < n ? none : tw_pack(0.f, tag);
    EE_TW_POLL(kB, src + at(min(base + k * kWG + static_cast<int>(threadIdx.x), n - 1)), true)
#pragma unroll
    for (int k = 0; k < kB; ++k) {
      const int i = base + k * kWG + static_cast<int>(threadIdx.x);
      if (i < n) xs[i] = tw_val(v[k]);
    }
  }
}

// ---------------------------------------------------------------------------
// reductions
// ---------------------------------------------------------------------------
// Reductions over a wave use DPP within rows of 16 lanes (a few cycles per
// step) and read the four row results with readlane, instead of a chain of
// LDS-routed lane shuffles (a round trip through LDS per step). Every lane
// gets the same, fixed-order result.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float readlane(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
// sum over aligned groups of 8 or 16 lanes
__device__ __forceinline__ float group_sum(float v, bool sixteen) {
  v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
  v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]: lane ^ 2
  v += dpp<0x141>(v);  // row_half_mirror: the other quad of the 8
  if (sixteen) v += dpp<0x140>(v);  // row_mirror: the other 8 of the 16
  return v;
}
__device__ __forceinline__ float group_max16(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  return fmaxf(v, dpp<0x140>(v));
}

__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum(v, true);
  return (readlane(v, 0) + readlane(v, 16)) + (readlane(v, 32) + readlane(v, 48));
}

__device__ __forceinline__ float wave_max(float v) {
  v = group_max16(v);
  return fmaxf(fmaxf(readlane(v, 0), readlane(v, 16)), fmaxf(readlane(v, 32), readlane(v, 48)));
}

template <int R>
__device__ __forceinline__ void wave_sum_n(float (&v)[R]) {
#pragma unroll
  for (int r = 0; r < R; ++r) v[r] = group_sum(v[r], true);
#pragma unroll
  for (int r = 0; r < R; ++r)
    v[r] = (readlane(v[r], 0) + readlane(v[r], 16)) + (readlane(v[r], 32) + readlane(v[r], 48));
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

// ---------------------------------------------------------------------------
// staging of activation vectors (written by other workgroups) into LDS:
// coherent 8-byte loads, up to 24 per thread in flight. n is even.
// ---------------------------------------------------------------------------
__device__ inline void stage_coh(const float* x, int n, float* xs) {
  const int n2 = n >> 1;
  uint64_t* dst = reinterpret_cast<uint64_t*>(xs);
  constexpr int kB = 24;  // loads per thread in flight: 12288 floats per round trip
  for (int base = 0; base < n2; base += kB * kWG) {
    uint64_t v[kB];
#pragma unroll
    for (int k = 0; k < kB; ++k) {
      const int i = base + k * kWG + static_cast<int>(threadIdx.x);
      v[k] = i < n2 ? ld_coh_u64(x + 2 * i) : 0ull;
    }
#pragma unroll
    for (int k = 0; k < kB; ++k) {
      const int i = base + k * kWG + static_cast<int>(threadIdx.x);
      if (i < n2) dst[i] = v[k];
    }
  }
}

// xs[i] = x[i] * rsqrt(mean(x^2) + eps) * (g ? g[i] : 1), x tagged words
// The gains of the thread's first kGR elements are requested before the
// input wait, so no global round trip follows it.
template <int kB = 8>
__device__ inline void rmsnorm_stage(const DevParams& p, const uint64_t* x, const float* __restrict__ g,
                                     int n, const Sync& sy, float* xs, float* red) {
  constexpr int kGR = 4;
  float gr[kGR];
#pragma unroll
  for (int j = 0; j < kGR; ++j) {
    const int i = static_cast<int>(threadIdx.x) + j * kWG;
    gr[j] = (g && i < n) ? g[i] : 1.f;
  }
  __syncthreads();  // xs may still be read by a previous phase
  tw_stage<kB>(p, x, n, sy.tin, sy.poll, xs);
  __syncthreads();
  float ss = 0.f;
  for (int i = threadIdx.x; i < n; i += kWG) ss = fmaf(xs[i], xs[i], ss);
  const float r = rsqrtf(block_sum(ss, red) / static_cast<float>(n) + p.eps);
#pragma unroll
  for (int j = 0; j < kGR; ++j) {
    const int i = static_cast<int>(threadIdx.x) + j * kWG;
    if (i < n) xs[i] = xs[i] * r * gr[j];
  }
  for (int i = static_cast<int>(threadIdx.x) + kGR * kWG; i < n; i += kWG) xs[i] = xs[i] * r * (g ? g[i] : 1.f);
  __syncthreads();
}

template <int kB = 8>
__device__ inline void copy_stage(const DevParams& p, const uint64_t* x, int n, const Sync& sy, float* xs) {
  __syncthreads();
  tw_stage<kB>(p, x, n, sy.tin, sy.poll, xs);
  __syncthreads();
}

// ---------------------------------------------------------------------------
// GEMV building block: R rows x CPL 16-byte chunks per lane held in
// registers. Lane `lane` owns chunks c0 + lane + 64k (k < CPL) below c1 of
// each row. load() issues every load before anything waits on them, so a wave
// can start fetching the next phase's weights before a grid barrier.
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

template <typename WT, int R, int CPL>
struct RowBlock {
  static constexpr int N = Elem<WT>::N;
  uint4 w[R][CPL];

  __device__ __forceinline__ void load(const WT* W, int64_t ld, int row0, int nr, int c0, int c1) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const uint4* row = reinterpret_cast<const uint4*>(W + static_cast<int64_t>(row0 + r) * ld);
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const int c = c0 + lane + 64 * k;
        w[r][k] = (r < nr && c < c1) ? row[c] : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  }

  // acc[r] = W[row r] . xs over this lane's chunks (partial: reduce over lanes after)
  __device__ __forceinline__ void dot(const float* xs, int nr, int c0, int c1, float (&acc)[R]) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int c = c0 + lane + 64 * k;
      if (c < c1) {
        float x[N];
        load_x<N>(xs, c, x);
#pragma unroll
        for (int r = 0; r < R; ++r)
          if (r < nr) acc[r] = fma_chunk<WT>(w[r][k], x, acc[r]);
      }
    }
  }

  // as dot(), with x scaled elementwise by g (global, read-only)
  __device__ __forceinline__ void dot_gain(const float* xs, const float* __restrict__ g, int nr, int c0,
                                           int c1, float (&acc)[R]) const {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int c = c0 + lane + 64 * k;
      if (c < c1) {
        float x[N];
        load_x<N>(xs, c, x);
#pragma unroll
        for (int e = 0; e < N; ++e) x[e] *= g[c * N + e];
#pragma unroll
        for (int r = 0; r < R; ++r)
          if (r < nr) acc[r] = fma_chunk<WT>(w[r][k], x, acc[r]);
      }
    }
  }
};

// Tiles of R rows x (at most 64*CPL) chunks covering rows [rb, re) and chunk
// range [cb, ce), row block by row block, double buffered: tile t+1 is loaded
// before tile t is consumed. Tile 0 must be loaded into `a` already (typically
// before a grid barrier wait). np = pieces per row block (the same for every
// wave that shares the row blocks). emit(row0, nrows, acc) receives each row
// block's wave-reduced dot products over [cb, ce).
template <typename WT, int R, int CPL>
struct Tiling {
  int rb, re, cb, ce, np;
  __device__ __forceinline__ int count() const { return ((re - rb + R - 1) / R) * np; }
  __device__ __forceinline__ int row(int t) const { return rb + (t / np) * R; }
  __device__ __forceinline__ int nrows(int t) const { return min(R, re - row(t)); }
  __device__ __forceinline__ int c0(int t) const { return cb + (t % np) * 64 * CPL; }
  __device__ __forceinline__ int c1(int t) const { return min(ce, c0(t) + 64 * CPL); }
  __device__ __forceinline__ void load(RowBlock<WT, R, CPL>& blk, const WT* W, int64_t ld, int t) const {
    blk.load(W, ld, row(t), nrows(t), c0(t), c1(t));
  }
};

template <typename WT, int R, int CPL, typename Emit>
__device__ __forceinline__ void stream_tiles(const WT* W, int64_t ld, const Tiling<WT, R, CPL>& tl,
                                             const float* xs, RowBlock<WT, R, CPL>& a,
                                             RowBlock<WT, R, CPL>& b, Emit&& emit, int preloaded = 1) {
  const int nt = tl.count();
  float tot[R];
#pragma unroll
  for (int r = 0; r < R; ++r) tot[r] = 0.f;
  auto consume = [&](const RowBlock<WT, R, CPL>& blk, int t) {
    float acc[R];
    blk.dot(xs, tl.nrows(t), tl.c0(t), tl.c1(t), acc);
#pragma unroll
    for (int r = 0; r < R; ++r) tot[r] += acc[r];
    if (t % tl.np == tl.np - 1) {
      wave_sum_n<R>(tot);
      emit(tl.row(t), tl.nrows(t), tot);
#pragma unroll
      for (int r = 0; r < R; ++r) tot[r] = 0.f;
    }
  };
  for (int t = 0; t < nt; t += 2) {
    if (t + 1 < nt && (t > 0 || preloaded < 2)) tl.load(b, W, ld, t + 1);
    consume(a, t);
    if (t + 1 >= nt) break;
    if (t + 2 < nt) tl.load(a, W, ld, t + 2);
    consume(b, t + 1);
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
// consecutive elements. q goes to its tagged vector; k and v go to the cache
// and, when kvnew is set, also (storage-rounded) to the tagged copy of this
// step's row that the attention phase reads.
// What the store of row pair r0 reads from global memory (the rotation of
// its RoPE pair, its cache row), gathered before the phase waits for its
// input so that no load round trip follows the dot product.
struct QkvPre {
  float c, s;    // cos / sin of the pair's angle at pos (q and k rows)
  int64_t off;   // cache offset of the row's (layer, position, kv head) (k and v rows)
};

__device__ inline QkvPre qkv_pre(const DevParams& p, int l, int pos, int r0) {
  const int AD = p.A * p.D, KD = p.K * p.D;
  QkvPre q{1.f, 0.f, 0};
  if (r0 < AD + KD) {
    const int head = r0 / p.D, rl = r0 - head * p.D, half = p.D >> 1;
    q.c = p.rope_cos[static_cast<int64_t>(pos) * half + (rl >> 1)];
    q.s = p.rope_sin[static_cast<int64_t>(pos) * half + (rl >> 1)];
    if (r0 >= AD) q.off = kv_offset(p, l, pos, head - p.A);
  } else {
    q.off = kv_offset(p, l, pos, (r0 - AD - KD) / p.D);
  }
  return q;
}

template <typename WT>
__device__ inline void store_qkv_pair(const DevParams& p, const QkvPre& pre, int r0, float x1, float x2,
                                      uint32_t tag, bool kvnew) {
  const int AD = p.A * p.D, KD = p.K * p.D;
  if (r0 < AD + KD) {
    const int head = r0 / p.D;
    const int rl = r0 - head * p.D;  // = 2i
    const float c = pre.c, s = pre.s;
    const float y1 = x1 * c - x2 * s;
    const float y2 = x2 * c + x1 * s;
    if (r0 < AD) {
      tw_store(p.q + r0, y1, tag);
      tw_store(p.q + r0 + 1, y2, tag);
    } else {
      WT* kp = static_cast<WT*>(p.kpool) + pre.off + rl;
      Elem<WT>::store_pair(kp, y1, y2);
      if (kvnew) {
        tw_store(p.kvnew + (r0 - AD), Elem<WT>::round(y1), tag);
        tw_store(p.kvnew + (r0 - AD) + 1, Elem<WT>::round(y2), tag);
      }
    }
  } else {
    const int j = r0 - AD - KD;
    const int d = j - (j / p.D) * p.D;
    WT* vp = static_cast<WT*>(p.vpool) + pre.off + d;
    Elem<WT>::store_pair(vp, x1, x2);
    if (kvnew) {
      tw_store(p.kvnew + KD + j, Elem<WT>::round(x1), tag);
      tw_store(p.kvnew + KD + j + 1, Elem<WT>::round(x2), tag);
    }
  }
}

// The input token of a step: forced, or emitted by the previous step (its
// tagged record inside a persistent launch, the control record otherwise).
__device__ inline int step_token(const DevParams& p, int step, const Sync& sy) {
  int tok;
  if (p.force_tok) tok = p.force_tok[step];
  else if (sy.poll && step > 0) tok = __float_as_int(tw_val(tw_wait(p, p.dec + 1, sy.tres, true)));
  else tok = ld_coh(&p.ctl->next_token);
  if (tok < 0 || tok >= p.V) {
    if (threadIdx.x == 0) atomicMax(&p.ctl->error, kErrToken);
    tok = 0;
  }
  return tok;
}

// The wave's index in the workgroup, as a wave-uniform (scalar) value: the
// row ranges, tile counts and loop bounds derived from it then live in scalar
// registers and branch on scalar conditions, instead of per-lane values whose
// loops and conditional tile loads compile to exec-mask sequences.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
}

// ---------------------------------------------------------------------------
// phase: RMSNorm + QKV projection + RoPE + KV append (one layer). Global wave
// gw owns row pair gw (+ total waves while rows remain). For layer 0 the input
// is the embedding row of the step's token, and workgroup 0 also initialises
// the residual stream h with it.
// ---------------------------------------------------------------------------
template <typename WT, int CPL>
struct QkvTask {
  RowBlock<WT, 2, CPL> blk;
  QkvPre pre;  // of the wave's first pair
  __device__ __forceinline__ void prefetch(const DevParams& p, int l, int pos, int wg) {
    const int pair = wg * kWaves + wave_id();
    if ((threadIdx.x & 63) == 0 && pair < (p.qkv_rows >> 1)) pre = qkv_pre(p, l, pos, 2 * pair);
    blk.load(static_cast<const WT*>(p.layers[l].wqkv), p.H, 2 * pair, pair < (p.qkv_rows >> 1) ? 2 : 0,
             0, p.H / Elem<WT>::N);
  }
};

template <typename WT, int CPL>
__device__ void phase_qkv(const DevParams& p, int l, int pos, int step, int wg, int nwg, float* xs,
                          float* red, QkvTask<WT, CPL>& t, const Sync& sy) {
  const int pairs = p.qkv_rows >> 1;
  if (wg * kWaves >= pairs) return;
  const LayerW lw = p.layers[l];
  if (l == 0) {
    // layer 0 starts from the token's embedding row; workgroup 0 also
    // publishes it as the residual stream h
    const int tok = step_token(p, step, sy);
    if (wg == 0 && threadIdx.x == 0 && p.hist_tok) p.hist_tok[pos] = tok;  // read after the launch
    const WT* e = static_cast<const WT*>(p.embed) + static_cast<int64_t>(tok) * p.H;
    __syncthreads();
    float ss = 0.f;
    for (int i = threadIdx.x; i < p.H; i += kWG) {
      const float v = Elem<WT>::load(e + i);
      xs[i] = v;
      ss = fmaf(v, v, ss);
      if (wg == 0) tw_store(p.h + i, v, sy.tout);
    }
    const float r = rsqrtf(block_sum(ss, red) / static_cast<float>(p.H) + p.eps);
    for (int i = threadIdx.x; i < p.H; i += kWG) xs[i] = xs[i] * r * lw.g_attn[i];
    __syncthreads();
    if (!sy.poll && wg == 0 && threadIdx.x == 0) st_coh(&p.ctl->exited, 0);
  } else {
    rmsnorm_stage(p, p.h, lw.g_attn, p.H, sy, xs, red);
  }
  const int nch = p.H / Elem<WT>::N;
  const int tw = nwg * kWaves;
  for (int pair = wg * kWaves + wave_id(); pair < pairs; pair += tw) {
    if (pair != wg * kWaves + wave_id())
      t.blk.load(static_cast<const WT*>(lw.wqkv), p.H, 2 * pair, 2, 0, nch);
    float acc[2];
    t.blk.dot(xs, 2, 0, nch, acc);
    wave_sum_n<2>(acc);
    if ((threadIdx.x & 63) == 0)
      store_qkv_pair<WT>(p, pair == wg * kWaves + wave_id() ? t.pre : qkv_pre(p, l, pos, 2 * pair), 2 * pair, acc[0],
                         acc[1], sy.tout, true);
  }
}

// ---------------------------------------------------------------------------
// phase: decode attention over positions 0..pos, grouped-query. Workgroup
// item = (kv head, pair of the query heads sharing it, split of kWaves
// attn_ppw(pos) positions); wave w of the item takes attn_ppw(pos) positions. Lane (sub, dl)
// of a wave holds 16-byte chunk dl of K and V rows sub + PPW k (LPP lanes per
// row, PPW rows per load, RPL rows per lane): a row's dot product with q is
// summed over its LPP lanes with DPP, the softmax statistics over the wave's
// rows stay in registers, and the weighted V rows are summed over the PPW row
// groups. The waves merge in LDS; with one split the item writes o directly,
// otherwise it publishes a partial (weighted V, max, sum of exp) as tagged
// words and the workgroup of the last split merges the others into o as they
// land (one kernel per operation: the last split to arrive merges). A
// workgroup runs its items in increasing order, so a merger only waits for
// items of lower index, which never wait for it. Splitting the query
// heads into pairs spreads the work over three times as many workgroups and
// keeps each partial small.
//
// Latency: every K and V row of a lane is loaded with independent loads. The
// rows of positions before pos were written in earlier steps, so the
// workgroup issues them (and the page-table lookups) before it waits for its
// input; only the row of position pos, written by the projection phase, is
// read after it (from its tagged copy).
// ---------------------------------------------------------------------------
// e^x as 2^(x log2 e) on the hardware base-2 exponential (v_exp_f32): within
// a few ulps, against a dozen instructions of the library routine's range
// reduction. Used on the attention softmax (arguments are scores minus their
// running maximum, <= 0; exp(-inf) = 0 for padded rows), in SiLU and in the
// vocabulary head's online softmax statistics.
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }

// Positions per wave of an item: kPosPerWave, or kPosPerWaveLong from
// kLongAttnFrom positions on, where twice the positions per item keep the
// items within one round of the workgroups and the merge within one LDS
// chunk (at 8192 positions: 198 items instead of 390, 33 records instead of
// 65). Every step picks it from its own position, identically in both
// programs.
__host__ __device__ inline int attn_ppw(int pos) { return pos >= kLongAttnFrom ? kPosPerWaveLong : kPosPerWave; }
__host__ __device__ inline int attn_split(int pos) { return kWaves * attn_ppw(pos); }
__host__ __device__ inline int attn_nsplit(int pos) { return (pos + attn_split(pos)) / attn_split(pos); }
__host__ __device__ inline int attn_pairs(int G) { return (G + 1) >> 1; }
constexpr int kAttnMergers = 4;  // merging splits per head pair in the long-context program
__host__ __device__ inline int attn_wave_floats(int D) {
  return 2 * kPosPerWaveLong + 2 * D + 4;  // offsets | weighted V of 2 heads | m0 m1 l0 l1
}
__host__ __device__ inline int attn_lds_floats(int D) { return 2 * D + kWaves * attn_wave_floats(D); }
__host__ __device__ inline int attn_rec_words(int D) { return 2 * D + 4; }  // partial record

// ---------------------------------------------------------------------------
// LDS layout: xs [vec] | red [64] (block sums, per-wave partial rows)
// ---------------------------------------------------------------------------
__host__ __device__ inline int lds_vec_floats(const DevParams& p) {
  int v = p.H;
  if (p.F > v) v = p.F;
  if (p.A * p.D > v) v = p.A * p.D;
  if (kWG * kStatFloats > v) v = kWG * kStatFloats;
  const int am = attn_lds_floats(p.D);
  if (am > v) v = am;
  return (v + 63) & ~63;
}

// Hides x from loop-invariant code motion: a value passed through here at the
// top of a loop body is unpacked inside the loop instead of being unpacked
// once into many more registers than the packed form takes.
__device__ __forceinline__ void keep_packed(uint4& x) {
  asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
}

// reductions over the PPW row groups of a wave (one value per group, read
// from the group's first lane); every lane gets the same result
// v summed over the lanes that share lane % LPP (LPP = 8 or 16): lane l gets
// the sum over l ^ 8 (LPP 8), l ^ 16 and l ^ 32 without LDS: a DPP rotate by
// 8 within 16-lane rows, then the gfx950 cross-row swaps. Every lane adds
// the same two values at each step, so all lanes hold the same bits.
__device__ __forceinline__ float add_swapped16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_swapped32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
template <int LPP>
__device__ __forceinline__ float sum_lanes_xor(float v) {
  static_assert(LPP == 8 || LPP == 16, "8 or 16 lanes per position");
  if constexpr (LPP == 8) v += dpp<0x128>(v);  // row_ror:8 = lane ^ 8 within the row
  return add_swapped32(add_swapped16(v));
}

template <int LPP>
__device__ __forceinline__ float groups_max(float v) {
  float m = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
#pragma unroll
  for (int r = 1; r < 64 / LPP; ++r)
    m = fmaxf(m, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), r * LPP)));
  return m;
}
template <int LPP>
__device__ __forceinline__ float groups_sum(float v) {
  float s = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
#pragma unroll
  for (int r = 1; r < 64 / LPP; ++r)
    s += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), r * LPP));
  return s;
}

// 16-byte chunks per cache row: 16 (256-byte rows) or 8 (128-byte rows)
template <typename WT>
__device__ __forceinline__ int attn_row_chunks(const DevParams& p) {
  return p.D / Elem<WT>::N;
}

// The K and V rows of one wave in registers; rows [0, nold) are positions
// before pos, and when has_new, row nold is position pos.
// pw positions per wave (attn_ppw of the step, at most CAP): the row slots
// past pw are neither loaded nor used. With CAP = kPosPerWave (steps below
// kLongAttnFrom only) pw is that constant.
template <typename WT, int CAP>
struct AttnTask {
  static constexpr int N = Elem<WT>::N;
  static constexpr int kRowsMax = CAP * 16 / 64;  // rows per lane at LPP = 16
  uint4 kr[kRowsMax], vr[kRowsMax];
  uint4 knew, vnew;  // row nold, in the lanes of row group nold % PPW
  int nold;
  int pw;
  bool has_new;

  __device__ __forceinline__ static int64_t* offw(const DevParams& p, float* lds) {
    return reinterpret_cast<int64_t*>(lds + 2 * p.D + wave_id() * attn_wave_floats(p.D));
  }
  // cache offsets of the wave's positions (up to pos) of item it, into LDS
  __device__ __forceinline__ void offsets(const DevParams& p, int l, int pos, int it, int nsplit,
                                          float* lds) {
    const int lane = threadIdx.x & 63;
    const int per_kvh = attn_pairs(p.G) * nsplit;
    const int kvh = it / per_kvh, sp = (it - kvh * per_kvh) % nsplit;
    const int ws0 = sp * kWaves * pw + wave_id() * pw;
    if (lane < pw && ws0 + lane <= pos) offw(p, lds)[lane] = kv_offset(p, l, ws0 + lane, kvh);
    __builtin_amdgcn_wave_barrier();
  }
  // Rows [0, n) into kr/vr. Slots of rows >= n load row n - 1 again (no
  // per-lane branches; their weight is zero), so every slot holds finite data.
  template <int LPP>
  __device__ __forceinline__ void load_old(const DevParams& p, const int64_t* ow, int n) {
    if (n <= 0) return;
    constexpr int PPW = 64 / LPP, RPL = CAP / PPW;
    const int lane = threadIdx.x & 63;
    const int sub = lane / LPP, dl = lane - sub * LPP;
    const WT* kp = static_cast<const WT*>(p.kpool);
    const WT* vp = static_cast<const WT*>(p.vpool);
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      if (CAP > kPosPerWave && PPW * k >= pw) break;
      const int64_t o = ow[min(sub + PPW * k, n - 1)] + dl * N;
      kr[k] = *reinterpret_cast<const uint4*>(kp + o);
      vr[k] = *reinterpret_cast<const uint4*>(vp + o);
    }
  }
  __device__ __forceinline__ void clear() {
#pragma unroll
    for (int k = 0; k < kRowsMax; ++k) kr[k] = vr[k] = make_uint4(0u, 0u, 0u, 0u);
    knew = vnew = make_uint4(0u, 0u, 0u, 0u);
    nold = 0;
    has_new = false;
  }
  // Before the input is ready: offsets and the rows of positions < pos of
  // the workgroup's first item (item it runs on workgroup nwg - 1 - it: the
  // last workgroups, which own no rows of the projections around attention).
  template <int LPP>
  __device__ __forceinline__ void prefetch(const DevParams& p, int l, int pos, int wg, int nwg, float* lds) {
    clear();
    pw = CAP > kPosPerWave ? attn_ppw(pos) : kPosPerWave;
    const int nsplit = attn_nsplit(pos);
    const int it = nwg - 1 - wg;
    if (it >= p.K * attn_pairs(p.G) * nsplit) return;
    const int ws0 = (it % nsplit) * kWaves * pw + wave_id() * pw;
    offsets(p, l, pos, it, nsplit, lds);
    nold = max(0, min(pw, pos - ws0));
    has_new = pos >= ws0 && pos < ws0 + pw;
    load_old<LPP>(p, offw(p, lds), nold);
  }
  // After the barrier: the row of position pos (first item only).
  template <int LPP>
  // (from the tagged copy the projection phase wrote along with the cache)
  __device__ __forceinline__ void load_new(const DevParams& p, int kvh, const Sync& sy) {
    if (!has_new) return;
    constexpr int PPW = 64 / LPP;
    const int lane = threadIdx.x & 63;
    const int sub = lane / LPP, dl = lane - sub * LPP;
    if (sub == nold % PPW) {
      const uint64_t* kw = p.kvnew + kvh * p.D + dl * N;
      float kf[N], vf[N];
      tw_read2<N>(p, kw, kw + p.K * p.D, sy.tin, sy.poll, kf, vf);
      knew = Elem<WT>::pack(kf);
      vnew = Elem<WT>::pack(vf);
    }
  }
  // the packed chunk of row slot k of this lane (the new row replaces the
  // slot it falls in); a select of values, never a store to a computed slot
  // (both operands are pinned to registers first: a select between two
  // members would otherwise become a load through a selected address, which
  // puts the whole task in private memory)
  template <int LPP>
  __device__ __forceinline__ uint4 krow(int k, int sub) {
    constexpr int PPW = 64 / LPP;
    uint4 a = kr[k], b = knew;
    keep_packed(a);
    keep_packed(b);
    return (has_new && k == nold / PPW && sub == nold % PPW) ? b : a;
  }
  template <int LPP>
  __device__ __forceinline__ uint4 vrow(int k, int sub) {
    constexpr int PPW = 64 / LPP;
    uint4 a = vr[k], b = vnew;
    keep_packed(a);
    keep_packed(b);
    return (has_new && k == nold / PPW && sub == nold % PPW) ? b : a;
  }
};

template <typename WT, int LPP, int CAP>
__device__ __forceinline__ void attn_item(const DevParams& p, int pos, int it, float* lds,
                                          AttnTask<WT, CAP>& t, const Sync& sy) {
  constexpr int N = Elem<WT>::N;
  constexpr int PPW = 64 / LPP, RPL = CAP / PPW;
  const int PW = CAP > kPosPerWave ? t.pw : kPosPerWave;
  const int T = pos + 1;
  const int nsplit = attn_nsplit(pos);
  const int G = p.G, D = p.D, GP = attn_pairs(G);
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int sub = lane / LPP, dl = lane - sub * LPP;
  const int kvh = it / (GP * nsplit), rem = it - kvh * GP * nsplit;
  const int gp = rem / nsplit, sp = rem - gp * nsplit;
  const int g0 = 2 * gp, g1 = min(g0 + 1, G - 1);  // g1 == g0: odd G, last pair
  const int WF = attn_wave_floats(D);
  float* qs = lds;  // [2][D] q of heads g0, g1 (unscaled)
  float* wb = lds + 2 * D + wave * WF;
  float* accw = wb + 2 * kPosPerWaveLong;  // [2][D]
  float* mlw = accw + 2 * D;           // m0 m1 l0 l1
  __shared__ int last_flag;

  const int ws0 = sp * kWaves * PW + wave * PW;
  const int wn = max(0, min(PW, T - ws0));  // positions of this wave
  const int tid = threadIdx.x;
  __syncthreads();
  if (tid < 2 * D)
    qs[tid] = tw_val(tw_wait(p, p.q + (kvh * G + (tid < D ? g0 : g1)) * D + (tid < D ? tid : tid - D),
                             sy.tin, sy.poll));
  t.template load_new<LPP>(p, kvh, sy);
  __syncthreads();

  if (wn > 0) {
    float qa[N], qb[N];
#pragma unroll
    for (int e = 0; e < N; ++e) {
      qa[e] = qs[dl * N + e];
      qb[e] = qs[D + dl * N + e];
    }
    float sa[RPL], sb[RPL];
    float ma = -INFINITY, mb = -INFINITY;
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      if (CAP > kPosPerWave && PPW * k >= PW) break;  // slots past the step's positions per wave
      uint4 kc = t.template krow<LPP>(k, sub);
      keep_packed(kc);
      float kf[N];
      Elem<WT>::unpack(kc, kf);
      float x = 0.f, y = 0.f;
#pragma unroll
      for (int e = 0; e < N; ++e) {
        x = fmaf(qa[e], kf[e], x);
        y = fmaf(qb[e], kf[e], y);
      }
      const bool valid = sub + PPW * k < wn;
      sa[k] = valid ? group_sum(x, LPP == 16) * p.attn_scale : -INFINITY;
      sb[k] = valid ? group_sum(y, LPP == 16) * p.attn_scale : -INFINITY;
      ma = fmaxf(ma, sa[k]);
      mb = fmaxf(mb, sb[k]);
    }
    ma = groups_max<LPP>(ma);
    mb = groups_max<LPP>(mb);
    float la = 0.f, lb = 0.f;
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      if (CAP > kPosPerWave && PPW * k >= PW) break;
      sa[k] = fexp(sa[k] - ma);  // exp(-inf) = 0 for rows past the wave's end
      sb[k] = fexp(sb[k] - mb);
      la += sa[k];
      lb += sb[k];
    }
    la = groups_sum<LPP>(la);
    lb = groups_sum<LPP>(lb);
    float aa[N], ab[N];
#pragma unroll
    for (int e = 0; e < N; ++e) aa[e] = ab[e] = 0.f;
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      if (CAP > kPosPerWave && PPW * k >= PW) break;
      uint4 vc = t.template vrow<LPP>(k, sub);
      keep_packed(vc);
      float vf[N];
      Elem<WT>::unpack(vc, vf);
#pragma unroll
      for (int e = 0; e < N; ++e) {
        aa[e] = fmaf(sa[k], vf[e], aa[e]);
        ab[e] = fmaf(sb[k], vf[e], ab[e]);
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) {
      aa[e] = sum_lanes_xor<LPP>(aa[e]);
      ab[e] = sum_lanes_xor<LPP>(ab[e]);
    }
    if (sub == 0) {
#pragma unroll
      for (int e = 0; e < N; ++e) {
        accw[dl * N + e] = aa[e];
        accw[D + dl * N + e] = ab[e];
      }
    }
    if (lane == 0) {
      mlw[0] = ma;
      mlw[1] = mb;
      mlw[2] = la;
      mlw[3] = lb;
    }
  }
  __syncthreads();
  // merge the waves of this item (fixed order): thread tid owns element
  // e = tid of [2][D] (head g0 + e / D, dimension e % D)
  const bool act = tid < 2 * D;
  const int hg = act ? tid / D : 0, dd = tid - hg * D;
  const bool dup = hg == 1 && g1 == g0;  // second head of an odd last pair
  const int nw = min(kWaves, (T - sp * kWaves * PW + PW - 1) / PW);
  float M = -INFINITY, den = 0.f, num = 0.f;
  {
    float mw[kWaves];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mw[w] = w < nw ? lds[2 * D + w * WF + 2 * kPosPerWaveLong + 2 * D + hg] : -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, mw[w]);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (w < nw) {
        const float* wb2 = lds + 2 * D + w * WF + 2 * kPosPerWaveLong;
        const float f = fexp(mw[w] - M);
        den = fmaf(f, wb2[2 * D + 2 + hg], den);
        num = fmaf(f, act ? wb2[tid] : 0.f, num);
      }
    }
  }
  uint64_t* outp = p.o + (kvh * G + g0 + hg) * D + dd;
  if (nsplit == 1) {
    if (act && !dup) tw_store(outp, num / den, sy.tout);
    return;
  }
  // partial records, tagged: [K][GP][max_splits][2D weighted V | m0 m1 | l0 l1]
  const int RS = attn_rec_words(D);
  uint64_t* recs = p.attn_part + (static_cast<int64_t>(kvh) * GP + gp) * p.max_splits * RS;
  const int cap = max(1, (lds_vec_floats(p) - 8) / (RS + 2));  // splits per merge chunk
  if constexpr (CAP > kPosPerWave) {
    // Many splits (the long-context program): every split publishes its
    // record and the last kAttnMergers splits each merge one slice of the 2D
    // elements, staging only that slice (and the head's max and sum) of every
    // record; one merger staging whole records would wait on several rounds
    // of loads. Same arithmetic, in the same chunks of splits, as the single
    // merger below. Only when every item has a workgroup of its own: a
    // merger here also waits for splits after its own, which in a second
    // round of items could wait for it.
    constexpr int MG = kAttnMergers;
    const int E = 2 * D / MG;           // elements per merger (within one head)
    const int RW = E + 2;               // staged words per record
    if (sy.poll && nsplit >= 2 * MG && nsplit * RW + 4 <= lds_vec_floats(p) &&
        p.K * GP * nsplit <= static_cast<int>(gridDim.x)) {
      uint64_t* r = recs + static_cast<int64_t>(sp) * RS;
      if (act) tw_store(r + tid, num, sy.tout);
      if (act && dd == 0) {
        tw_store(r + 2 * D + hg, M, sy.tout);
        tw_store(r + 2 * D + 2 + hg, den, sy.tout);
      }
      const int mk = nsplit - 1 - sp;  // merger index
      if (mk >= MG) return;
      const int e0 = mk * E, mh = e0 / D;  // the slice's first element and its head
      __syncthreads();  // LDS may still be read (wave records)
      float* rl = lds;  // [nsplit][RW]: the slice's weighted V, then the head's max and sum
      tw_gather<8>(p, recs, nsplit * RW, [&](int i) {
        const int s2 = i / RW, j = i - s2 * RW;
        return static_cast<int64_t>(s2) * RS + (j < E ? e0 + j : 2 * D + (j - E) * 2 + mh);
      }, sy.tout, sy.poll, rl);
      __syncthreads();
      if (tid < E) {
        const int e = e0 + tid, dm = e - mh * D;
        float Mr = -INFINITY, Dr = 0.f, Nr = 0.f;
        for (int c0 = 0; c0 < nsplit; c0 += cap) {
          const int ns = min(cap, nsplit - c0);
          float cm = Mr;
          for (int s2 = 0; s2 < ns; ++s2) cm = fmaxf(cm, rl[(c0 + s2) * RW + E]);
          const float sc = fexp(Mr - cm);
          float dn = Dr * sc;
          Nr *= sc;
          for (int s2 = 0; s2 < ns; ++s2) {
            const float* rr = rl + (c0 + s2) * RW;
            const float f = fexp(rr[E] - cm);
            dn = fmaf(f, rr[E + 1], dn);
            Nr = fmaf(f, rr[tid], Nr);
          }
          Mr = cm;
          Dr = dn;
        }
        const bool dup_m = mh == 1 && g1 == g0;
        if (!dup_m) tw_store(p.o + (kvh * G + g0 + mh) * D + dm, Nr * (1.f / Dr), sy.tout);
      }
      return;
    }
  }
  const bool merger = sy.poll && sp == nsplit - 1;
  if (!merger) {
    uint64_t* r = recs + static_cast<int64_t>(sp) * RS;
    if (act) tw_store(r + tid, num, sy.tout);
    if (act && dd == 0) {
      tw_store(r + 2 * D + hg, M, sy.tout);
      tw_store(r + 2 * D + 2 + hg, den, sy.tout);
    }
    if (sy.poll) return;
    wait_stores();
    __syncthreads();
    if (tid == 0) {
      const uint32_t old = __hip_atomic_fetch_add(&p.counters->attn[kvh * GP + gp][0], 1u,
                                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last_flag = (old == static_cast<uint32_t>(nsplit - 1));
    }
    __syncthreads();
    if (!last_flag) return;
  }
  // Merge in chunks of splits staged into LDS, in split order: per head a
  // running max and sum (held by the head's first thread), per element a
  // running weighted V. The merger (the last split) writes its own record
  // into its slot instead of reading it back, so both programs do the same
  // arithmetic in the same order.
  float Mr = -INFINITY, Dr = 0.f, Nr = 0.f;
  float* rl = lds;                 // [cap][RS]
  float* wts = lds + cap * RS;     // [cap][2] split weights
  float* hsc = wts + 2 * cap;      // [2] rescale of the running values, then [2] 1 / sum
  for (int c0 = 0; c0 < nsplit; c0 += cap) {
    const int ns = min(cap, nsplit - c0);
    const bool own = merger && c0 + ns == nsplit;  // this chunk holds the merger's split
    __syncthreads();  // LDS may still be read (wave records, previous chunk)
    tw_stage<12>(p, recs + static_cast<int64_t>(c0) * RS, (ns - (own ? 1 : 0)) * RS, sy.tout, sy.poll, rl);
    if (own) {
      float* r = rl + (ns - 1) * RS;
      if (act) r[tid] = num;
      if (act && dd == 0) {
        r[2 * D + hg] = M;
        r[2 * D + 2 + hg] = den;
      }
    }
    __syncthreads();
    if (act && dd == 0) {
      float cm = Mr;
      for (int s2 = 0; s2 < ns; ++s2) cm = fmaxf(cm, rl[s2 * RS + 2 * D + hg]);
      const float sc = fexp(Mr - cm);  // 0 while nothing has been merged yet
      float dn = Dr * sc;
      for (int s2 = 0; s2 < ns; ++s2) {
        const float f = fexp(rl[s2 * RS + 2 * D + hg] - cm);
        wts[s2 * 2 + hg] = f;
        dn = fmaf(f, rl[s2 * RS + 2 * D + 2 + hg], dn);
      }
      hsc[hg] = sc;
      Mr = cm;
      Dr = dn;
    }
    __syncthreads();
    if (act) {
      Nr *= hsc[hg];
      for (int s2 = 0; s2 < ns; ++s2) Nr = fmaf(wts[s2 * 2 + hg], rl[s2 * RS + tid], Nr);
    }
  }
  __syncthreads();
  if (act && dd == 0) hsc[2 + hg] = 1.f / Dr;
  __syncthreads();
  if (act && !dup) tw_store(outp, Nr * hsc[2 + hg], sy.tout);
  if (!sy.poll && tid == 0)
    __hip_atomic_store(&p.counters->attn[kvh * GP + gp][0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The first item of the workgroup uses the rows t prefetched; further items
// (more than one per workgroup only when the items outnumber the workgroups)
// load theirs when they start.
template <typename WT, int LPP, int CAP>
__device__ __forceinline__ void phase_attn(const DevParams& p, int l, int pos, int wg, int nwg,
                                           float* lds, AttnTask<WT, CAP>& t, const Sync& sy) {
  const int nsplit = attn_nsplit(pos);
  const int items = p.K * attn_pairs(p.G) * nsplit;
  const int first = nwg - 1 - wg;
  for (int it = first; it < items; it += nwg) {
    if (it != first) {
      __syncthreads();  // offsets of the previous item may still be read
      t.offsets(p, l, pos, it, nsplit, lds);
      const int pw = CAP > kPosPerWave ? t.pw : kPosPerWave;
      const int ws0 = (it % nsplit) * kWaves * pw + wave_id() * pw;
      t.nold = max(0, min(pw, pos - ws0));
      t.has_new = pos >= ws0 && pos < ws0 + pw;  // read from its tagged copy
      t.template load_old<LPP>(p, AttnTask<WT, CAP>::offw(p, lds), t.nold);
    }
    attn_item<WT, LPP, CAP>(p, pos, it, lds, t, sy);
  }
}

// The attention phase with the row layout (lanes per cache row); after the
// prefetch, before the wait, `mark` runs (the timeline stamp of the
// persistent program).
template <typename WT, int LPP, int CAP, typename Mark>
__device__ __forceinline__ void attn_run(const DevParams& p, int l, int pos, int wg, int nwg, float* lds,
                                         const Sync& sy, Mark&& mark) {
  AttnTask<WT, CAP> t;
  t.template prefetch<LPP>(p, l, pos, wg, nwg, lds);
  mark(0u);
  phase_attn<WT, LPP, CAP>(p, l, pos, wg, nwg, lds, t, sy);
}

// CAP: the most positions per wave this program's steps use (kPosPerWave
// when every step lies below kLongAttnFrom)
template <typename WT, int CAP, typename Mark>
__device__ __forceinline__ void attn_dispatch(const DevParams& p, int l, int pos, int wg, int nwg, float* lds,
                                              const Sync& sy, Mark&& mark) {
  if (attn_row_chunks<WT>(p) == 16) attn_run<WT, 16, CAP>(p, l, pos, wg, nwg, lds, sy, mark);
  else attn_run<WT, 8, CAP>(p, l, pos, wg, nwg, lds, sy, mark);
}

// ---------------------------------------------------------------------------
// phase: one row per wave, out[r] = W[r] . x (+ bias) or out[r] += W[r] . x.
// Used for Wo (residual) and the readout (bias).
// ---------------------------------------------------------------------------
template <typename WT, int CPL>
struct RowTask {
  RowBlock<WT, 1, CPL> blk;
  __device__ __forceinline__ void prefetch(const WT* W, int rows, int cols, int wg) {
    const int r = wg * kWaves + wave_id();
    blk.load(W, cols, r, r < rows ? 1 : 0, 0, cols / Elem<WT>::N);
  }
};

template <typename WT, int CPL>
__device__ void phase_rows(const DevParams& p, const WT* W, int rows, int cols, const uint64_t* x,
                           uint64_t* out, const float* bias, int residual, int wg, int nwg, float* xs,
                           RowTask<WT, CPL>& t, const Sync& sy) {
  if (wg * kWaves >= rows) return;
  const int r0 = wg * kWaves + wave_id();
  // the residual of the wave's first row is read before the input is staged
  float prev0 = 0.f;
  if (residual && (threadIdx.x & 63) == 0 && r0 < rows) prev0 = tw_val(tw_wait(p, out + r0, sy.tres, sy.poll));
  else if (bias && (threadIdx.x & 63) == 0 && r0 < rows) prev0 = bias[r0];  // requested before the input wait
  copy_stage(p, x, cols, sy, xs);
  const int nch = cols / Elem<WT>::N;
  const int tw = nwg * kWaves;
  for (int r = r0; r < rows; r += tw) {
    if (r != r0) t.blk.load(W, cols, r, 1, 0, nch);
    float acc[1];
    t.blk.dot(xs, 1, 0, nch, acc);
    acc[0] = wave_sum(acc[0]);
    if ((threadIdx.x & 63) == 0) {
      float prev = r == r0 ? prev0 : (bias ? bias[r] : 0.f);
      if (residual && r != r0) prev = tw_val(tw_wait(p, out + r, sy.tres, sy.poll));
      tw_store(out + r, prev + acc[0], sy.tout);
    }
  }
}

// ---------------------------------------------------------------------------
// phase: RMSNorm + gate/up projection + SiLU(gate) * up. Interleaved rows
// (2j = gate j, 2j+1 = up j). Global wave gw owns the contiguous output range
// [gw F / W, (gw+1) F / W), streamed in blocks of two outputs.
// ---------------------------------------------------------------------------
constexpr int kRS = 4;  // rows per streamed block

// Gate/up rows per block: two blocks, both requested before the input wait,
// hold all of a wave's 8-9 rows at the 1.5B shape; wide rows (CPL 4) keep
// blocks of 4 within the register budget.
template <int CPL>
constexpr int gu_rows() { return CPL >= 4 ? 4 : 6; }

__device__ __forceinline__ int gu_begin(const DevParams& p, int gw, int tw) {
  return static_cast<int>(static_cast<int64_t>(p.F) * gw / tw);
}

template <typename WT, int CPL>
struct GateUpTask {
  RowBlock<WT, gu_rows<CPL>(), CPL> a, b;
  __device__ __forceinline__ static Tiling<WT, gu_rows<CPL>(), CPL> tiling(const DevParams& p, int wg, int nwg) {
    const int tw = nwg * kWaves, gw = wg * kWaves + wave_id();
    return Tiling<WT, gu_rows<CPL>(), CPL>{2 * gu_begin(p, gw, tw), 2 * gu_begin(p, gw + 1, tw), 0,
                                p.H / Elem<WT>::N, 1};
  }
  __device__ __forceinline__ void prefetch(const DevParams& p, int l, int wg, int nwg) {
    const auto tl = tiling(p, wg, nwg);
    const WT* W = static_cast<const WT*>(p.layers[l].wgu);
    if (tl.count() > 0) tl.load(a, W, p.H, 0);
    if (tl.count() > 1) tl.load(b, W, p.H, 1);
  }
};

__device__ inline float silu(float x) { return x / (1.f + fexp(-x)); }

template <typename WT, int CPL>
__device__ void phase_gateup(const DevParams& p, int l, int wg, int nwg, float* xs, float* red,
                             GateUpTask<WT, CPL>& t, const Sync& sy) {
  const int tw = nwg * kWaves;
  const int gw0 = wg * kWaves;
  if (gu_begin(p, gw0 + kWaves, tw) == gu_begin(p, gw0, tw)) return;
  const LayerW lw = p.layers[l];
  rmsnorm_stage(p, p.h, lw.g_mlp, p.H, sy, xs, red);
  uint64_t* a_out = p.a;
  stream_tiles<WT, gu_rows<CPL>(), CPL>(static_cast<const WT*>(lw.wgu), p.H, GateUpTask<WT, CPL>::tiling(p, wg, nwg),
                             xs, t.a, t.b, [&](int r0, int nr, const float(&acc)[gu_rows<CPL>()]) {
                              if ((threadIdx.x & 63) == 0) {
#pragma unroll
                                for (int i = 0; i < gu_rows<CPL>() / 2; ++i)
                                  if (2 * i < nr) tw_store(a_out + r0 / 2 + i, silu(acc[2 * i]) * acc[2 * i + 1], sy.tout);
                              }
                            }, 2);
}

// ---------------------------------------------------------------------------
// phase: h += W_d a. Workgroup wg owns rows [wg H / nwg, (wg+1) H / nwg); its
// waves split the F dimension into kWaves contiguous chunk ranges and stream
// tiles of kRS rows x 64*CPL chunks; per row block the partial sums of the
// waves meet in LDS.
// ---------------------------------------------------------------------------
template <typename WT, int CPL>
struct DownTask {
  RowBlock<WT, kRS, CPL> a, b;
  uint64_t hraw;  // residual word h[rb + threadIdx.x] of the workgroup's rows (first kWG rows)
  __device__ __forceinline__ static Tiling<WT, kRS, CPL> tiling(const DevParams& p, int wg, int nwg) {
    const int nch = p.F / Elem<WT>::N;
    const int longest = (nch + kWaves - 1) / kWaves;
    return Tiling<WT, kRS, CPL>{static_cast<int>(static_cast<int64_t>(p.H) * wg / nwg),
                                static_cast<int>(static_cast<int64_t>(p.H) * (wg + 1) / nwg),
                                nch * wave_id() / kWaves, nch * (wave_id() + 1) / kWaves,
                                max(1, (longest + 64 * CPL - 1) / (64 * CPL))};
  }
  // Before the input is ready: the residual words (h is last written by the
  // output projection, before the gate/up phase), then the first two tiles.
  // Nothing waits here: the residual's tag is checked once a is staged (a
  // wait now would also wait for the tiles requested after it).
  __device__ __forceinline__ void prefetch(const DevParams& p, int l, int wg, int nwg) {
    const auto tl = tiling(p, wg, nwg);
    const WT* W = static_cast<const WT*>(p.layers[l].wd);
    const int r = tl.rb + static_cast<int>(threadIdx.x);
    hraw = r < tl.re ? ld_coh_u64(p.h + r) : 0ull;
    if (tl.count() > 0) tl.load(a, W, p.F, 0);
    if (tl.count() > 1) tl.load(b, W, p.F, 1);
  }
};

template <typename WT, int CPL>
__device__ void phase_down(const DevParams& p, int l, int wg, int nwg, float* xs, float* red,
                           DownTask<WT, CPL>& t, const Sync& sy) {
  const auto tl = DownTask<WT, CPL>::tiling(p, wg, nwg);
  if (tl.rb >= tl.re) return;
  copy_stage<18>(p, p.a, p.F, sy, xs);
  const int wave = wave_id();
  const int tid = threadIdx.x;
  float hres = 0.f;
  if (tl.rb + tid < tl.re)
    hres = tw_val(tw_ok(t.hraw, sy.tres) ? t.hraw : tw_wait(p, p.h + tl.rb + tid, sy.tres, sy.poll));
  uint64_t* h = p.h;
  stream_tiles<WT, kRS, CPL>(static_cast<const WT*>(p.layers[l].wd), p.F, tl, xs, t.a, t.b,
                             [&](int r0, int nr, const float(&acc)[kRS]) {
                               if ((tid & 63) == 0) {
#pragma unroll
                                 for (int i = 0; i < kRS; ++i) red[wave * kRS + i] = acc[i];
                               }
                               __syncthreads();
                               // the thread that holds row r's residual updates it
                               const int i = tid - (r0 - tl.rb);
                               if (i >= 0 && i < nr) {
                                 float sum = 0.f;
                                 for (int w = 0; w < kWaves; ++w) sum += red[w * kRS + i];
                                 tw_store(h + r0 + i, hres + sum, sy.tout);
                               } else if (r0 - tl.rb + nr > kWG && tid < nr && r0 - tl.rb + tid >= kWG) {
                                 float sum = 0.f;
                                 for (int w = 0; w < kWaves; ++w) sum += red[w * kRS + tid];
                                 const float prev = tw_val(tw_wait(p, h + r0 + tid, sy.tres, sy.poll));
                                 tw_store(h + r0 + tid, prev + sum, sy.tout);
                               }
                               __syncthreads();
                             }, 2);
}

// ---------------------------------------------------------------------------
// phase: head = RMSNorm(src; g_final) -> unembedding -> online (max, argmax,
// sum exp, second max) over the vocabulary, never writing logits (unless a
// debug buffer is given). Each workgroup owns a contiguous row range split in
// contiguous eighths, one per wave, streamed in blocks of kRS rows; the
// workgroup writes one partial and the last workgroup merges the partials
// with a fixed tree, takes the gate decision (readout) or the final token,
// and emits.
// ---------------------------------------------------------------------------
struct Stat {
  float m;    // max logit
  float s;    // sum of exp(logit - m)
  float m2;   // second largest logit (equal to m on ties)
  int idx;    // argmax, lowest index among ties
  float t;    // sum of exp(logit - m) * (logit - m), for the entropy
  float a;    // sum of exp(logit - m) over the tokens ahead of a reference token
};

__device__ inline Stat stat_empty() { return Stat{-INFINITY, 0.f, -INFINITY, 0x7fffffff, 0.f, 0.f}; }

// ahead: the token sorts before the reference token (higher logit, or equal
// logit and lower id)
__device__ inline void stat_push(Stat& st, float v, int r, bool ahead) {
  if (v > st.m) {
    const float sc = fexp(st.m - v);
    st.t = st.s > 0.f ? sc * (st.t + (st.m - v) * st.s) : 0.f;
    st.a = st.a * sc + (ahead ? 1.f : 0.f);
    st.s = st.s * sc + 1.f;
    st.m2 = st.m;
    st.m = v;
    st.idx = r;
  } else {
    const float e = fexp(v - st.m);
    st.s += e;
    st.t = fmaf(e, v - st.m, st.t);
    if (ahead) st.a += e;
    st.m2 = fmaxf(st.m2, v);
  }
}

__device__ inline Stat stat_merge(Stat a, Stat b) {
  if (b.s == 0.f) return a;
  if (a.s == 0.f) return b;
  const bool bw = b.m > a.m || (b.m == a.m && b.idx < a.idx);
  Stat w = bw ? b : a;
  const Stat o = bw ? a : b;
  const float sc = fexp(o.m - w.m);
  w.t = w.t + sc * (o.t + (o.m - w.m) * o.s);
  w.a = w.a + o.a * sc;
  w.s = w.s + o.s * sc;
  w.m2 = fmaxf(w.m2, o.m);
  return w;
}

__device__ inline void stat_put(float* d, const Stat& st) {
  d[0] = st.m;
  d[1] = st.s;
  d[2] = st.m2;
  d[3] = __int_as_float(st.idx);
  d[4] = st.t;
  d[5] = st.a;
}
__device__ inline Stat stat_get(const float* d) {
  return Stat{d[0], d[1], d[2], __float_as_int(d[3]), d[4], d[5]};
}

// The confidence the gate compares with tau (Section 10 names three softmax
// measures): 0 the best token's probability 1/s; 1 its margin over the
// second best, (1 - exp(m2 - m)) / s; 2 the negative entropy
// sum p log p = t/s - log s.
__device__ inline float stat_confidence(const Stat& st, int measure) {
  if (measure == 1) return (1.f - expf(st.m2 - st.m)) / st.s;
  if (measure == 2) return st.t / st.s - logf(st.s);
  return 1.f / st.s;
}

__device__ __forceinline__ int head_row(const DevParams& p, int wg, int nwg, int wave) {
  // workgroup wg owns rows [V wg / nwg, V (wg+1) / nwg); wave w the w-th eighth of them
  const int64_t rb = static_cast<int64_t>(p.V) * wg / nwg;
  const int64_t re = static_cast<int64_t>(p.V) * (wg + 1) / nwg;
  return static_cast<int>(rb + (re - rb) * wave / kWaves);
}

template <typename WT, int CPL, int R = kRS>
struct HeadTask {
  RowBlock<WT, R, CPL> a, b;
  __device__ __forceinline__ static Tiling<WT, R, CPL> tiling(const DevParams& p, int wg, int nwg) {
    return Tiling<WT, R, CPL>{head_row(p, wg, nwg, wave_id()), head_row(p, wg, nwg, wave_id() + 1), 0,
                              p.H / Elem<WT>::N, 1};
  }
  __device__ __forceinline__ void prefetch(const DevParams& p, int wg, int nwg) {
    const auto tl = tiling(p, wg, nwg);
    const WT* W = static_cast<const WT*>(p.embed);
    if (tl.count() > 0) tl.load(a, W, p.H, 0);
    if (tl.count() > 1) tl.load(b, W, p.H, 1);
  }
};

template <typename WT, int CPL, int R = kRS>
__device__ void phase_head(const DevParams& p, int readout, int step, int wg, int nwg, float* xs,
                           float* red, HeadTask<WT, CPL, R>& t, const Sync& sy) {
  rmsnorm_stage(p, readout ? p.z : p.h, p.g_final, p.H, sy, xs, red);
  float* dbg = readout ? p.dbg_logits_r : p.dbg_logits_f;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  // Nucleus membership of the readout's token under the full head (Section
  // 2): the mass of the tokens ahead of it. Its logit is computed the way
  // the scan computes row nj (same lanes, same order), so the token is never
  // ahead of itself.
  __shared__ int sh_nj;
  __shared__ float sh_lj;
  int nj = -1;
  float lj = 0.f;
  if (!readout && p.nucleus && p.exit_layer > 0) {
    if (threadIdx.x == 0)
      sh_nj = sy.poll ? __float_as_int(tw_val(tw_wait(p, p.dec + 4, sy.tres, true))) : ld_coh(&p.ctl->readout_token);
    __syncthreads();
    nj = sh_nj;
    if (wave == 0) {
      const int nch = p.H / Elem<WT>::N;
      RowBlock<WT, 1, CPL> rj;
      rj.load(static_cast<const WT*>(p.embed), p.H, nj, 1, 0, nch);
      float acc[1], tot[1] = {0.f};
      rj.dot(xs, 1, 0, nch, acc);
      tot[0] += acc[0];
      wave_sum_n<1>(tot);
      if (lane == 0) sh_lj = tot[0];
    }
    __syncthreads();
    lj = sh_lj;
  }
  Stat st = stat_empty();
  stream_tiles<WT, R, CPL>(static_cast<const WT*>(p.embed), p.H, HeadTask<WT, CPL, R>::tiling(p, wg, nwg),
                           xs, t.a, t.b, [&](int r0, int nr, const float(&acc)[R]) {
#pragma unroll
                              for (int r = 0; r < R; ++r)
                                if (r < nr)
                                  stat_push(st, acc[r], r0 + r,
                                            nj >= 0 && (acc[r] > lj || (acc[r] == lj && r0 + r < nj)));
                              if (dbg && lane == 0)
                                for (int r = 0; r < nr; ++r) dbg[r0 + r] = acc[r];
                            }, 2);
  __shared__ int last_flag;
  float* stl = xs;  // the normalised vector is no longer needed: kWG * kStatFloats floats
  __syncthreads();
  if (lane == 0) stat_put(stl + wave * kStatFloats, st);
  __syncthreads();
  if (threadIdx.x == 0) {
    Stat tt = stat_empty();
    for (int w = 0; w < kWaves; ++w) tt = stat_merge(tt, stat_get(stl + w * kStatFloats));
    float* part = p.head_part + static_cast<int64_t>(wg) * kStatFloats;
    st_coh2(part, tt.m, tt.s);
    st_coh2(part + 2, tt.m2, __int_as_float(tt.idx));
    st_coh2(part + 4, tt.t, tt.a);
    wait_stores();
    const uint32_t old = __hip_atomic_fetch_add(&p.counters->head[0], 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    last_flag = (old == sy.cbase + static_cast<uint32_t>(nwg - 1));
  }
  __syncthreads();
  if (!last_flag) return;
  // the partials of up to 4 * kWG workgroups are loaded before any is merged
  Stat tt = stat_empty();
  for (int i0 = 0; i0 < nwg; i0 += 4 * kWG) {
    uint64_t a[4], b[4], c[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = i0 + k * kWG + static_cast<int>(threadIdx.x);
      const float* part = p.head_part + static_cast<int64_t>(min(i, nwg - 1)) * kStatFloats;
      a[k] = ld_coh_u64(part);
      b[k] = ld_coh_u64(part + 2);
      c[k] = ld_coh_u64(part + 4);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (i0 + k * kWG + static_cast<int>(threadIdx.x) < nwg)
        tt = stat_merge(tt, Stat{__uint_as_float(static_cast<uint32_t>(a[k])),
                                 __uint_as_float(static_cast<uint32_t>(a[k] >> 32)),
                                 __uint_as_float(static_cast<uint32_t>(b[k])),
                                 static_cast<int>(static_cast<uint32_t>(b[k] >> 32)),
                                 __uint_as_float(static_cast<uint32_t>(c[k])),
                                 __uint_as_float(static_cast<uint32_t>(c[k] >> 32))});
    }
  }
  stat_put(stl + threadIdx.x * kStatFloats, tt);
  __syncthreads();
  for (int stride = kWG / 2; stride > 0; stride >>= 1) {
    if (static_cast<int>(threadIdx.x) < stride)
      stat_put(stl + threadIdx.x * kStatFloats,
               stat_merge(stat_get(stl + threadIdx.x * kStatFloats),
                          stat_get(stl + (threadIdx.x + stride) * kStatFloats)));
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const Stat fin = stat_get(stl);
    const int idx = fin.idx;
    const float conf = stat_confidence(fin, p.conf_measure);
    StepCtl* c = p.ctl;
    if (!sy.poll)
      __hip_atomic_store(&p.counters->head[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (readout) {
      const int would = conf > p.tau;
      const int fe = p.force_exit ? p.force_exit[step] : -1;
      const int ex = fe < 0 ? would : fe;
      // the gate record every workgroup reads: exited, token, confidence, decision
      tw_store(p.dec + 2, conf, sy.tout);
      tw_store(p.dec + 3, __int_as_float(would), sy.tout);
      tw_store(p.dec + 4, __int_as_float(idx), sy.tout);
      if (ex) tw_store(p.dec + 1, __int_as_float(idx), sy.tout);
      tw_store(p.dec + 0, __int_as_float(ex), sy.tout);
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
          if (p.ring_would) p.ring_would[step] = would;
        }
      }
    } else {
      const int gated = p.exit_layer > 0;
      tw_store(p.dec + 1, __int_as_float(idx), sy.tout);
      st_coh(&c->full_token, idx);
      st_coh(&c->conf_full, conf);
      st_coh(&c->next_token, idx);
      if (p.ring_tok) {
        float rconf = conf;
        int rwould = 0;
        if (gated && sy.poll) {  // this step's gate record (tag sy.tres)
          rconf = tw_val(tw_wait(p, p.dec + 2, sy.tres, true));
          rwould = __float_as_int(tw_val(tw_wait(p, p.dec + 3, sy.tres, true)));
        } else if (gated) {
          rconf = ld_coh(&c->conf);
          rwould = ld_coh(&c->would_exit);
        }
        p.ring_tok[step] = idx;
        p.ring_exit[step] = 0;
        p.ring_conf[step] = rconf;
        if (p.ring_would) p.ring_would[step] = rwould;
        if (nj >= 0 && p.ring_mass) p.ring_mass[step] = fin.a / fin.s;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// phase: KV-absence fill after an exit. For every skipped layer l (exit_layer
// .. L-1, 0-based): a = RMSNorm(h_exit; g_attn[l]); K_l[pos] = RoPE(W_k,l a),
// V_l[pos] = W_v,l a. Global wave gw owns row pairs gw, gw + W, ... over the
// layers' k and v rows; the normalisation is staged once without gain and
// each layer's gain is applied chunk by chunk.
// ---------------------------------------------------------------------------
template <typename WT, int CPL>
__device__ void phase_fill(const DevParams& p, int pos, int wg, int nwg, float* xs, float* red,
                           const Sync& sy) {
  const int KD = p.K * p.D;  // row pairs per layer (k and v rows: 2*KD)
  const int total = (p.L - p.exit_layer) * KD;
  if (wg * kWaves >= total) return;
  rmsnorm_stage(p, p.h_exit, nullptr, p.H, sy, xs, red);
  const int nch = p.H / Elem<WT>::N;
  const int tw = nwg * kWaves;
  RowBlock<WT, 2, CPL> blk;
  for (int q = wg * kWaves + wave_id(); q < total; q += tw) {
    const int l = p.exit_layer + q / KD;
    const int r0 = p.A * p.D + 2 * (q - (q / KD) * KD);
    const LayerW lw = p.layers[l];
    blk.load(static_cast<const WT*>(lw.wqkv), p.H, r0, 2, 0, nch);
    float acc[2];
    blk.dot_gain(xs, lw.g_attn, 2, 0, nch, acc);
    wave_sum_n<2>(acc);
    if ((threadIdx.x & 63) == 0) store_qkv_pair<WT>(p, qkv_pre(p, l, pos, r0), r0, acc[0], acc[1], sy.tout, false);
  }
}

// Lazy fill (persistent kernel): the exit-layer states of np exited steps
// (slots 0..np-1 of h_exit, tags ptag) are projected through every skipped
// layer's key and value rows at once: each row pair is loaded once and
// applied to every pending state, with the arithmetic of phase_fill, so the
// cache entries are the ones an eager fill writes.
template <typename WT, int CPL>
__device__ void phase_fill_batch(const DevParams& p, int np, const int* ppos, const uint32_t* ptag, int wg,
                                 int nwg, float* xs, float* red, const Sync& sy) {
  const int KD = p.K * p.D;
  const int total = (p.L - p.exit_layer) * KD;
  if (wg * kWaves >= total) return;
  for (int k = 0; k < np; ++k) {
    const Sync sk{sy.poll, ptag[k], 0u, sy.tout, 0u};
    rmsnorm_stage(p, p.h_exit + static_cast<int64_t>(k) * p.H, nullptr, p.H, sk, xs + k * p.H, red);
  }
  const int nch = p.H / Elem<WT>::N;
  const int tw = nwg * kWaves;
  RowBlock<WT, 2, CPL> blk;
  for (int q = wg * kWaves + wave_id(); q < total; q += tw) {
    const int l = p.exit_layer + q / KD;
    const int r0 = p.A * p.D + 2 * (q - (q / KD) * KD);
    const LayerW lw = p.layers[l];
    blk.load(static_cast<const WT*>(lw.wqkv), p.H, r0, 2, 0, nch);
    for (int k = 0; k < np; ++k) {
      float acc[2];
      blk.dot_gain(xs + k * p.H, lw.g_attn, 2, 0, nch, acc);
      wave_sum_n<2>(acc);
      if ((threadIdx.x & 63) == 0)
        store_qkv_pair<WT>(p, qkv_pre(p, l, ppos[k], r0), r0, acc[0], acc[1], sy.tout, false);
    }
  }
}

// readout: z = W_r h + b_r; workgroup 0 also keeps h as h_exit (in slot).
template <typename WT, int CPL>
__device__ void phase_readout(const DevParams& p, int wg, int nwg, float* xs, RowTask<WT, CPL>& t,
                              const Sync& sy, int slot = 0) {
  if (wg == 0) {
    uint64_t* hx = p.h_exit + static_cast<int64_t>(slot) * p.H;
    for (int i = threadIdx.x; i < p.H; i += kWG)
      tw_store(hx + i, tw_val(tw_wait(p, p.h + i, sy.tin, sy.poll)), sy.tout);
  }
  phase_rows<WT, CPL>(p, static_cast<const WT*>(p.ro_w), p.H, p.H, p.h, p.z, p.ro_b, 0, wg, nwg, xs, t, sy);
}

size_t lds_bytes(const DevParams& p) {
  return static_cast<size_t>(lds_vec_floats(p) + 64) * sizeof(float);
}

int fill_batch_slots(const DevParams& p) {
  const int k = lds_vec_floats(p) / p.H;  // normalised exit-layer states staged side by side
  return k < kMaxPending ? k : kMaxPending;
}

struct Lds {
  float* xs;
  float* red;
};

__device__ inline Lds lds_carve(const DevParams& p, float* smem) {
  return Lds{smem, smem + lds_vec_floats(p)};
}

// ---------------------------------------------------------------------------
// one-kernel-per-operation drivers
// ---------------------------------------------------------------------------
enum OpKind : int {
  kOpQkv = 0, kOpAttn, kOpWo, kOpGateUp, kOpDown, kOpReadout, kOpHeadR, kOpHeadF, kOpFill
};

template <typename WT, int CPL, int OP>
__global__ __launch_bounds__(kWG) void k_op(DevParams p, int l, int pos, int step, int skip_if_exited) {
  extern __shared__ float smem[];
  if (skip_if_exited && ld_coh(&p.ctl->exited)) return;
  const Lds s = lds_carve(p, smem);
  const int wg = blockIdx.x, nwg = gridDim.x;
  const Sync sy{false, 0u, 0u, 0u, 0u};  // kernel boundaries order the operations
  if constexpr (OP == kOpQkv) {
    QkvTask<WT, CPL> t;
    t.prefetch(p, l, pos, wg);
    phase_qkv<WT, CPL>(p, l, pos, step, wg, nwg, s.xs, s.red, t, sy);
  }
  if constexpr (OP == kOpAttn) attn_dispatch<WT, kPosPerWaveLong>(p, l, pos, wg, nwg, s.xs, sy, [](uint32_t) {});
  if constexpr (OP == kOpWo) {
    const WT* W = static_cast<const WT*>(p.layers[l].wo);
    RowTask<WT, CPL> t;
    t.prefetch(W, p.H, p.A * p.D, wg);
    phase_rows<WT, CPL>(p, W, p.H, p.A * p.D, p.o, p.h, nullptr, 1, wg, nwg, s.xs, t, sy);
  }
  if constexpr (OP == kOpGateUp) {
    GateUpTask<WT, CPL> t;
    t.prefetch(p, l, wg, nwg);
    phase_gateup<WT, CPL>(p, l, wg, nwg, s.xs, s.red, t, sy);
  }
  if constexpr (OP == kOpDown) {
    DownTask<WT, CPL> t;
    t.prefetch(p, l, wg, nwg);
    phase_down<WT, CPL>(p, l, wg, nwg, s.xs, s.red, t, sy);
  }
  if constexpr (OP == kOpReadout) {
    RowTask<WT, CPL> t;
    t.prefetch(static_cast<const WT*>(p.ro_w), p.H, p.H, wg);
    phase_readout<WT, CPL>(p, wg, nwg, s.xs, t, sy);
  }
  if constexpr (OP == kOpHeadR || OP == kOpHeadF) {
    HeadTask<WT, CPL> t;
    t.prefetch(p, wg, nwg);
    phase_head<WT, CPL>(p, OP == kOpHeadR, step, wg, nwg, s.xs, s.red, t, sy);
  }
  if constexpr (OP == kOpFill)
    if (ld_coh(&p.ctl->exited)) phase_fill<WT, CPL>(p, pos, wg, nwg, s.xs, s.red, sy);
}

static int op_grid(const DevParams& p, int op, int pos, int head_wgs) {
  switch (op) {
    case kOpQkv: return ((p.qkv_rows >> 1) + kWaves - 1) / kWaves;
    case kOpAttn: return p.K * attn_pairs(p.G) * attn_nsplit(pos);
    case kOpWo:
    case kOpReadout: return (p.H + kWaves - 1) / kWaves;
    case kOpGateUp: return (p.F + kWaves * 4 - 1) / (kWaves * 4);
    case kOpDown: return (p.H + 5) / 6;
    case kOpHeadR:
    case kOpHeadF: return head_wgs;
    case kOpFill: {
      const int total = (p.L - p.exit_layer) * p.K * p.D;
      return total > 0 ? (total + kWaves - 1) / kWaves : 1;
    }
  }
  return 1;
}

template <typename WT, int CPL>
static hipError_t op(const DevParams& p, int kind, int l, int pos, int step, int skip, int head_wgs,
                     hipStream_t s) {
  const int grid = op_grid(p, kind, pos, head_wgs);
  const size_t lds = lds_bytes(p);
  switch (kind) {
#define EE_OP_CASE(K)                                                                             \
  case K:                                                                                         \
    hipLaunchKernelGGL((k_op<WT, CPL, K>), dim3(grid), dim3(kWG), lds, s, p, l, pos, step, skip); \
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

template <typename WT, int CPL>
static hipError_t layer_ops(const DevParams& p, int l, int pos, int step, int skip, int hw,
                            hipStream_t s) {
  hipError_t e;
  if ((e = op<WT, CPL>(p, kOpQkv, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  if ((e = op<WT, CPL>(p, kOpAttn, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  if ((e = op<WT, CPL>(p, kOpWo, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  if ((e = op<WT, CPL>(p, kOpGateUp, l, pos, step, skip, hw, s)) != hipSuccess) return e;
  return op<WT, CPL>(p, kOpDown, l, pos, step, skip, hw, s);
}

// One decode step (or one prompt position when emit_head == 0) per op.
template <typename WT, int CPL>
static hipError_t step_per_op(const DevParams& p, int pos, int step, int emit_head, int hw,
                              hipStream_t s) {
  hipError_t e;
  const int Le = p.exit_layer;
  for (int l = 0; l < Le; ++l)
    if ((e = layer_ops<WT, CPL>(p, l, pos, step, 0, hw, s)) != hipSuccess) return e;
  if (Le > 0) {
    if ((e = op<WT, CPL>(p, kOpReadout, 0, pos, step, 0, hw, s)) != hipSuccess) return e;
    if ((e = op<WT, CPL>(p, kOpHeadR, 0, pos, step, 0, hw, s)) != hipSuccess) return e;
    if ((e = op<WT, CPL>(p, kOpFill, 0, pos, step, 0, hw, s)) != hipSuccess) return e;
  }
  for (int l = Le; l < p.L; ++l)
    if ((e = layer_ops<WT, CPL>(p, l, pos, step, Le > 0, hw, s)) != hipSuccess) return e;
  if (emit_head) return op<WT, CPL>(p, kOpHeadF, 0, pos, step, Le > 0, hw, s);
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// persistent cooperative kernel: n whole decode steps in one launch
// ---------------------------------------------------------------------------
// Two-level grid barrier, split in arrive and wait so that a workgroup can
// issue the next phase's weight loads in between. Epochs count barriers of
// the launch; wait() for an epoch already reached returns at once. The wait
// is bounded: on time-out the abort flag is raised and every later wait
// returns at once, so the grid always drains.
__device__ inline void bar_arrive(const DevParams& p, uint32_t& epoch, int wg, int nwg) {
  ++epoch;
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int g = wg & (kBarGroups - 1);
    const uint32_t per = static_cast<uint32_t>((nwg - g + kBarGroups - 1) / kBarGroups);
    const uint32_t old = __hip_atomic_fetch_add(&p.counters->group[g][0], 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    if (old == per * epoch - 1) {
      const uint32_t ngroups = static_cast<uint32_t>(min(kBarGroups, nwg));
      const uint32_t o2 = __hip_atomic_fetch_add(&p.counters->top[0], 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
      if (o2 == ngroups * epoch - 1)
        __hip_atomic_store(&p.counters->gen[0], epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

__device__ inline void bar_wait(const DevParams& p, uint32_t epoch) {
  if (threadIdx.x == 0) {
    uint32_t* gen = &p.counters->gen[0];
    const uint64_t t0 = wall_clock64();
    while (true) {
      const uint32_t v = __hip_atomic_load(gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (static_cast<int32_t>(v - epoch) >= 0) break;
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

// The steps of the persistent program. Tags holds, identically in every
// workgroup (the control flow is uniform), the tag of the latest version of
// each vector and the arrivals counted so far on the last-arriver counters.
struct Tags {
  uint32_t ep;                 // phases run in this launch; phase e writes tag e
  uint32_t h, q, o, a, z, hx;  // latest version of each vector
  uint32_t gate;               // latest gate record (readout head)
  uint32_t tok;                // record holding the next input token
  uint32_t heads;              // head phases run
};

__device__ __forceinline__ void tl_mark(const DevParams& p, uint32_t idx) {
  if (p.timeline && blockIdx.x == 0 && threadIdx.x == 0 && static_cast<int>(idx) < p.timeline_cap)
    p.timeline[idx] = wall_clock64();
}

// Each step reads the workgroup index through an opaque scalar move: values
// derived from it (row ranges, weight pointers) are then computed inside the
// step rather than hoisted out of the step and layer loops, where the
// invariants of every phase would otherwise stay live together and exhaust
// the registers.
__device__ __forceinline__ int opaque_wg() {
  int v;
  asm volatile("s_mov_b32 %0, %1" : "=s"(v) : "s"(static_cast<int>(blockIdx.x)));
  return v;
}
#define EE_PHASE_FN template <typename WT, int CPL> __device__ __forceinline__ void

EE_PHASE_FN run_qkv(const DevParams& p, int l, int pos, int step, float* smem, Tags& tg) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  QkvTask<WT, CPL> t;
  t.prefetch(p, l, pos, wg);
  const uint32_t E = ++tg.ep;
  tl_mark(p, 2 * E);
  phase_qkv<WT, CPL>(p, l, pos, step, wg, gridDim.x, s.xs, s.red, t, Sync{true, tg.h, tg.tok, E, 0u});
  tl_mark(p, 2 * E + 1);
  tg.q = E;
  if (l == 0) tg.h = E;
}

template <typename WT, int CPL, int CAP>
__device__ __forceinline__ void run_attn(const DevParams& p, int l, int pos, float* smem, Tags& tg) {
  const int wg = opaque_wg();
  // the prefetch writes row offsets into LDS, which waves of this workgroup
  // may still be reading as the projection phase's input
  __syncthreads();
  const uint32_t E = ++tg.ep;
  const Sync sy{true, tg.q, 0u, E, 0u};
  attn_dispatch<WT, CAP>(p, l, pos, wg, gridDim.x, smem, sy, [&](uint32_t) { tl_mark(p, 2 * E); });
  tl_mark(p, 2 * E + 1);
  tg.o = E;
}

// The gate/up tiles are requested here too, before the wait for the
// attention output: most workgroups have no attention item and would leave
// HBM idle while the attention workgroups finish. Not at long contexts
// (early_gu false): there the attention's K and V rows are a large read of
// their own, which the gate/up tiles would delay; they are requested when
// the gate/up phase starts instead.
EE_PHASE_FN run_wo(const DevParams& p, int l, float* smem, Tags& tg, GateUpTask<WT, CPL>& gu, bool early_gu) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  const WT* W = static_cast<const WT*>(p.layers[l].wo);
  RowTask<WT, CPL> t;
  t.prefetch(W, p.H, p.A * p.D, wg);
  if (early_gu) gu.prefetch(p, l, wg, gridDim.x);
  const uint32_t E = ++tg.ep;
  tl_mark(p, 2 * E);
  phase_rows<WT, CPL>(p, W, p.H, p.A * p.D, p.o, p.h, nullptr, 1, wg, gridDim.x, s.xs, t,
                      Sync{true, tg.o, tg.h, E, 0u});
  tl_mark(p, 2 * E + 1);
  tg.h = E;
}

EE_PHASE_FN run_gateup(const DevParams& p, int l, float* smem, Tags& tg, GateUpTask<WT, CPL>& t, bool early_gu) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  if (!early_gu) t.prefetch(p, l, wg, gridDim.x);
  const uint32_t E = ++tg.ep;
  tl_mark(p, 2 * E);
  phase_gateup<WT, CPL>(p, l, wg, gridDim.x, s.xs, s.red, t, Sync{true, tg.h, 0u, E, 0u});
  tl_mark(p, 2 * E + 1);
  tg.a = E;
}

EE_PHASE_FN run_down(const DevParams& p, int l, float* smem, Tags& tg) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  const uint32_t E = ++tg.ep;
  const Sync sy{true, tg.a, tg.h, E, 0u};
  DownTask<WT, CPL> t;
  t.prefetch(p, l, wg, gridDim.x);
  tl_mark(p, 2 * E);
  phase_down<WT, CPL>(p, l, wg, gridDim.x, s.xs, s.red, t, sy);
  tl_mark(p, 2 * E + 1);
  tg.h = E;
}

EE_PHASE_FN run_readout(const DevParams& p, float* smem, Tags& tg, int slot) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  RowTask<WT, CPL> t;
  t.prefetch(static_cast<const WT*>(p.ro_w), p.H, p.H, wg);
  const uint32_t E = ++tg.ep;
  tl_mark(p, 2 * E);
  phase_readout<WT, CPL>(p, wg, gridDim.x, s.xs, t, Sync{true, tg.h, 0u, E, 0u}, slot);
  tl_mark(p, 2 * E + 1);
  tg.z = E;
  tg.hx = E;
}

EE_PHASE_FN run_head(const DevParams& p, int readout, int step, float* smem, Tags& tg) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  HeadTask<WT, CPL> t;
  t.prefetch(p, wg, gridDim.x);
  const uint32_t E = ++tg.ep;
  tl_mark(p, 2 * E);
  phase_head<WT, CPL>(p, readout, step, wg, gridDim.x, s.xs, s.red, t,
                      Sync{true, readout ? tg.z : tg.h, tg.gate, E, tg.heads * gridDim.x});
  tl_mark(p, 2 * E + 1);
  ++tg.heads;
  if (readout) tg.gate = E;
}

EE_PHASE_FN run_fill(const DevParams& p, int pos, float* smem, Tags& tg) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  const uint32_t E = ++tg.ep;
  tl_mark(p, 2 * E);
  phase_fill<WT, CPL>(p, pos, wg, gridDim.x, s.xs, s.red, Sync{true, tg.hx, 0u, E, 0u});
  tl_mark(p, 2 * E + 1);
}

EE_PHASE_FN run_fill_batch(const DevParams& p, int np, const int* ppos, const uint32_t* ptag, float* smem,
                           Tags& tg) {
  const int wg = opaque_wg();
  const Lds s = lds_carve(p, smem);
  const uint32_t E = ++tg.ep;
  tl_mark(p, 2 * E);
  phase_fill_batch<WT, CPL>(p, np, ppos, ptag, wg, gridDim.x, s.xs, s.red, Sync{true, 0u, 0u, E, 0u});
  tl_mark(p, 2 * E + 1);
}
#undef EE_PHASE_FN

template <typename WT, int CPL, int CAP>
__device__ __forceinline__ void run_layer(const DevParams& p, int l, int pos, int step, float* smem,
                                          Tags& tg) {
  run_qkv<WT, CPL>(p, l, pos, step, smem, tg);
  run_attn<WT, CPL, CAP>(p, l, pos, smem, tg);
  GateUpTask<WT, CPL> gu;
  const bool early_gu = !(CAP > kPosPerWave && pos >= kLongAttnFrom);
  run_wo<WT, CPL>(p, l, smem, tg, gu, early_gu);
  run_gateup<WT, CPL>(p, l, smem, tg, gu, early_gu);
  run_down<WT, CPL>(p, l, smem, tg);
}

// Parameters of the persistent kernel live in constant memory, one slot per
// context: fields are read with scalar loads, and the kernel never copies the
// parameter block into private memory (which a by-value argument of this size
// in a kernel this large would cost).
__constant__ DevParams c_params[kParamSlots];

// prefill != 0: prompt positions, ungated, head only at the last position.
// One loop over the layers (a single inlined copy of the layer code); the
// readout and the gate run after layer exit_layer, and an exit leaves the
// loop for the KV fill of the remaining layers. Every step ends with a grid
// barrier: the next step reads KV rows this step wrote (the fill's included),
// and with forced tokens nothing else orders the two steps.
// With the lazy fill an exit only records its position and keeps its
// exit-layer state in the next h_exit slot; the pending positions are filled
// together before the first layer above exit_layer runs (then a grid barrier
// orders the new rows before that layer's attention reads them), when the
// slots are full, and before the launch ends.
// CAP: attention positions per wave the launch may use (kPosPerWave when
// every position of the launch lies below kLongAttnFrom).
template <typename WT, int CPL, int CAP>
__global__ __launch_bounds__(kWG) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_decode_persistent(
    int slot, int pos0, int n, int prefill) {
  extern __shared__ float smem[];
  __shared__ int sh_exited;
  __shared__ int sh_pend_pos[kMaxPending];
  __shared__ uint32_t sh_pend_tag[kMaxPending];
  const DevParams& p = c_params[slot];
  Tags tg{};
  uint32_t bep = 0;
  const int Le = p.exit_layer;
  const bool lazy = !prefill && p.lazy_fill > 1 && Le > 0 && Le < p.L;  // lazy_fill = slots
  int npend = 0;
  for (int i = 0; i < n; ++i) {
    if (aborted(p)) break;
    const int pos = pos0 + i;
    int exited = 0;
    for (int l = 0; l < p.L; ++l) {
      run_layer<WT, CPL, CAP>(p, l, pos, i, smem, tg);
      if (l + 1 == Le) {
        run_readout<WT, CPL>(p, smem, tg, lazy ? npend : 0);
        run_head<WT, CPL>(p, 1, i, smem, tg);
        __syncthreads();
        if (threadIdx.x == 0) sh_exited = __float_as_int(tw_val(tw_wait(p, p.dec, tg.gate, true)));
        __syncthreads();
        exited = sh_exited;
        if (exited) {
          tg.tok = tg.gate;
          break;
        }
        if (npend > 0) {  // the layers above read the pending positions' rows
          run_fill_batch<WT, CPL>(p, npend, sh_pend_pos, sh_pend_tag, smem, tg);
          npend = 0;
          bar_arrive(p, bep, blockIdx.x, gridDim.x);
          bar_wait(p, bep);
        }
      }
    }
    if (exited) {
      if (lazy) {
        __syncthreads();
        if (threadIdx.x == 0) {
          sh_pend_pos[npend] = pos;
          sh_pend_tag[npend] = tg.hx;
        }
        __syncthreads();
        if (++npend == p.lazy_fill) {
          run_fill_batch<WT, CPL>(p, npend, sh_pend_pos, sh_pend_tag, smem, tg);
          npend = 0;
        }
      } else if (Le < p.L) {
        run_fill<WT, CPL>(p, pos, smem, tg);
      }
    } else if (!prefill || i == n - 1) {
      run_head<WT, CPL>(p, 0, i, smem, tg);
      tg.tok = tg.ep;
    }
    bar_arrive(p, bep, blockIdx.x, gridDim.x);
    bar_wait(p, bep);
  }
  if (npend > 0 && !aborted(p)) run_fill_batch<WT, CPL>(p, npend, sh_pend_pos, sh_pend_tag, smem, tg);
}

// Launch state of the persistent kernel: barrier and last-arriver counters,
// and every tagged word (tag 0 is never written inside a launch).
__global__ __launch_bounds__(kWG) void k_reset_state(Counters* c, uint64_t* tw, int64_t nw) {
  const int t = threadIdx.x;
  if (blockIdx.x == 0) {
    if (t < kBarGroups) c->group[t][0] = 0u;
    if (t < 64) c->attn[t][0] = 0u;
    if (t == 0) {
      c->top[0] = 0u;
      c->gen[0] = 0u;
      c->head[0] = 0u;
    }
  }
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kWG + t; i < nw; i += static_cast<int64_t>(gridDim.x) * kWG)
    tw[i] = 0ull;
}

// The per-call fields of the step record (everything but next_token, the
// first step's input), cleared by a kernel rather than a memset node.
__global__ __launch_bounds__(64) void k_clear_step(StepCtl* c) {
  if (threadIdx.x == 0) {
    c->exited = 0;
    c->would_exit = 0;
    c->readout_token = 0;
    c->full_token = 0;
    c->conf = 0.f;
    c->conf_full = 0.f;
    c->error = 0;
    c->abort = 0u;
  }
}

hipError_t launch_clear_step(StepCtl* c, hipStream_t s) {
  hipLaunchKernelGGL(k_clear_step, dim3(1), dim3(64), 0, s, c);
  return hipGetLastError();
}

__global__ __launch_bounds__(kWG) void k_tag_vec(uint64_t* dst, const float* src, int n) {
  for (int i = blockIdx.x * kWG + threadIdx.x; i < n; i += gridDim.x * kWG) dst[i] = tw_pack(src[i], 0u);
}

__global__ __launch_bounds__(kWG) void k_untag(float* dst, const uint64_t* src, int n) {
  for (int i = blockIdx.x * kWG + threadIdx.x; i < n; i += gridDim.x * kWG) dst[i] = tw_val(src[i]);
}

// ---------------------------------------------------------------------------
// Library-resident scratch for the allocation-free decode entry point: the
// working set of a decode call (tagged activation words, attention and head
// partial records, barrier counters) placed in a fixed device array instead
// of memory the context allocates. Each device holds its own copy at its own
// address; host code never passes the array's name to a kernel, only the
// address hipGetSymbolAddress returns for the device that was current.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};
}  // namespace

hipError_t scratch_address(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // the caller makes the device current
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[device] = a;
  }
  *out = g_scratch_addr[device];
  return hipSuccess;
}

hipError_t launch_untag(float* dst, const uint64_t* src, int n, hipStream_t s) {
  hipLaunchKernelGGL(k_untag, dim3(8), dim3(kWG), 0, s, dst, src, n);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// host dispatch over (storage type, chunks per lane)
// ---------------------------------------------------------------------------
int chunks_per_lane(const DevParams& p, int wbf16) {
  const int nch = p.H / (wbf16 ? 8 : 4);
  return (nch + 63) / 64;
}

template <typename F>
static hipError_t dispatch(int wbf16, int cpl, F&& f) {
  if (wbf16) {
    switch (cpl) {
      case 1: return f(uint16_t{}, std::integral_constant<int, 1>{});
      case 2: return f(uint16_t{}, std::integral_constant<int, 2>{});
      case 3: return f(uint16_t{}, std::integral_constant<int, 3>{});
      case 4: return f(uint16_t{}, std::integral_constant<int, 4>{});
    }
  } else {
    switch (cpl) {
      case 1: return f(float{}, std::integral_constant<int, 1>{});
      case 2: return f(float{}, std::integral_constant<int, 2>{});
    }
  }
  return hipErrorInvalidValue;
}

// one kernel per operation relies on counters that start at zero (a
// persistent launch leaves them counting)
static hipError_t reset_counters(const DevParams& p, hipStream_t s) {
  hipLaunchKernelGGL(k_reset_state, dim3(1), dim3(kWG), 0, s, p.counters, p.tw_all, int64_t(0));
  return hipGetLastError();
}

hipError_t launch_decode_per_op(const DevParams& p, int wbf16, int pos0, int n, int head_wgs,
                                hipStream_t s) {
  const hipError_t e0 = reset_counters(p, s);
  if (e0 != hipSuccess) return e0;
  return dispatch(wbf16, chunks_per_lane(p, wbf16), [&](auto wt, auto cpl) {
    using WT = decltype(wt);
    for (int i = 0; i < n; ++i) {
      const hipError_t e = step_per_op<WT, decltype(cpl)::value>(p, pos0 + i, i, 1, head_wgs, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  });
}

hipError_t launch_prefill_per_op(const DevParams& p, int wbf16, int pos0, const int32_t* d_tokens,
                                 int n, int head_wgs, hipStream_t s) {
  DevParams q = p;
  q.exit_layer = 0;
  q.force_tok = d_tokens;
  q.force_exit = nullptr;
  const hipError_t e0 = reset_counters(p, s);
  if (e0 != hipSuccess) return e0;
  return dispatch(wbf16, chunks_per_lane(p, wbf16), [&](auto wt, auto cpl) {
    using WT = decltype(wt);
    for (int i = 0; i < n; ++i) {
      const hipError_t e =
          step_per_op<WT, decltype(cpl)::value>(q, pos0 + i, i, i == n - 1, head_wgs, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  });
}

hipError_t launch_head_eval(const DevParams& p, int wbf16, const float* d_x, int readout, int head_wgs,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_tag_vec, dim3(8), dim3(kWG), 0, s, p.h, d_x, p.H);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = reset_counters(p, s);
  if (e != hipSuccess) return e;
  return dispatch(wbf16, chunks_per_lane(p, wbf16), [&](auto wt, auto cpl) {
    using WT = decltype(wt);
    constexpr int C = decltype(cpl)::value;
    if (readout) {
      const hipError_t e2 = op<WT, C>(p, kOpReadout, 0, 0, 0, 0, head_wgs, s);
      if (e2 != hipSuccess) return e2;
    }
    return op<WT, C>(p, readout ? kOpHeadR : kOpHeadF, 0, 0, 0, 0, head_wgs, s);
  });
}

template <int CAP>
static const void* persistent_fn_cap(int wbf16, int cpl) {
  if (wbf16) {
    switch (cpl) {
      case 1: return reinterpret_cast<const void*>(&k_decode_persistent<uint16_t, 1, CAP>);
      case 2: return reinterpret_cast<const void*>(&k_decode_persistent<uint16_t, 2, CAP>);
      case 3: return reinterpret_cast<const void*>(&k_decode_persistent<uint16_t, 3, CAP>);
      case 4: return reinterpret_cast<const void*>(&k_decode_persistent<uint16_t, 4, CAP>);
    }
  } else {
    switch (cpl) {
      case 1: return reinterpret_cast<const void*>(&k_decode_persistent<float, 1, CAP>);
      case 2: return reinterpret_cast<const void*>(&k_decode_persistent<float, 2, CAP>);
    }
  }
  return nullptr;
}

// positions [pos0, end): the program whose attention items take as many
// positions per wave as the launch's last position needs
static const void* persistent_fn(int wbf16, int cpl, int end) {
  return end > kLongAttnFrom ? persistent_fn_cap<kPosPerWaveLong>(wbf16, cpl)
                             : persistent_fn_cap<kPosPerWave>(wbf16, cpl);
}

static hipError_t persistent(const PersistentLaunch& L, int pos0, int n, int prefill) {
  const DevParams& p = *L.params_host;
  const void* fn = persistent_fn(L.wbf16, chunks_per_lane(p, L.wbf16), pos0 + n);
  if (!fn || L.slot < 0 || L.slot >= kParamSlots) return hipErrorInvalidValue;
  hipError_t e = hipMemcpyToSymbolAsync(HIP_SYMBOL(c_params), L.params_host, sizeof(DevParams),
                                        sizeof(DevParams) * L.slot, hipMemcpyHostToDevice, L.stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_reset_state, dim3(16), dim3(kWG), 0, L.stream, p.counters, p.tw_all, p.tw_words);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int slot = L.slot;
  void* args[] = {&slot, &pos0, &n, &prefill};
  return hipLaunchCooperativeKernel(fn, dim3(L.nwg), dim3(kWG), args, static_cast<unsigned>(L.lds),
                                    L.stream);
}

hipError_t launch_decode_persistent(const PersistentLaunch& L, int pos0, int n) {
  return persistent(L, pos0, n, 0);
}

hipError_t launch_prefill_persistent(const PersistentLaunch& L, int pos0, int n) {
  return persistent(L, pos0, n, 1);
}

int persistent_max_wgs_per_cu(const DevParams& p, int wbf16, size_t lds) {
  // both programs: the grid must fit either
  int nb = 0, nl = 0;
  const void* fn = persistent_fn_cap<kPosPerWave>(wbf16, chunks_per_lane(p, wbf16));
  const void* fl = persistent_fn_cap<kPosPerWaveLong>(wbf16, chunks_per_lane(p, wbf16));
  if (!fn || !fl || hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, kWG, lds) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&nl, fl, kWG, lds) != hipSuccess)
    return 0;
  return nb < nl ? nb : nl;
}

}  // namespace ee
