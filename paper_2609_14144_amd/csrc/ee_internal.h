// Internal types shared by the runtime (ee_api.hip) and the kernels
// (ee_kernels.hip). Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ee {

constexpr int kWG = 512;               // threads per workgroup, every kernel
constexpr int kWaves = kWG / 64;       // 64-wide wavefronts per workgroup
constexpr int kPosPerWave = 16;             // attention positions per wave
constexpr int kPosPerWaveLong = 32;         // ... from kLongAttnFrom positions on
constexpr int kLongAttnFrom = 4096;
constexpr int kAttnSplit = kWaves * kPosPerWave;  // positions per attention work item (the smaller)
constexpr int kMaxGroup = 8;           // max query heads per KV head
constexpr int kMaxHeadDim = 256;
constexpr int kBarGroups = 8;          // first level of the grid barrier (one per XCD)
constexpr int kParamSlots = 16;        // persistent-kernel parameter blocks per device
constexpr int kMaxPending = 8;         // exit-layer states a lazy fill batches at most
constexpr size_t kScratchBytes = size_t(4) << 20;  // library-resident scratch per device
constexpr int kMaxDevices = 64;
constexpr int kStatFloats = 6;         // a head partial (max, sum, second max, argmax, entropy term, mass ahead)

// Per-layer device pointers, repacked layouts:
//   wqkv [(A + 2K) * D][H]: q rows, then k rows, then v rows. Within every q
//        and k head the rows are pair-interleaved: row 2i is the original row
//        i and row 2i+1 the original row i + D/2, so one wave computes both
//        halves of a rotate-half RoPE pair.
//   wo   [H][A*D]
//   wgu  [2F][H]: row 2j = gate row j, row 2j+1 = up row j.
//   wd   [H][F]
struct LayerW {
  const void* wqkv;
  const void* wo;
  const void* wgu;
  const void* wd;
  const float* g_attn;
  const float* g_mlp;
};

// Device-side control record of the step being run (one per context).
struct StepCtl {
  int32_t next_token;     // input of the next step (last emitted token)
  int32_t exited;         // branch taken by the current step
  int32_t would_exit;     // gate decision before forcing
  int32_t readout_token;
  int32_t full_token;
  float conf;             // readout confidence
  float conf_full;        // full head confidence
  int32_t error;          // nonzero: device-side failure (see kErr*)
  uint32_t abort;         // set when a bounded wait times out; everything drains
  uint32_t pad[7];
};

enum : int32_t { kErrNone = 0, kErrBarrier = 1, kErrToken = 2, kErrWait = 3 };

// Grid barrier / last-arriver counters. Each lives on its own 256-byte line.
// Barrier: workgroup wg arrives on group[wg % 8]; the last arrival of a group
// arrives on top; the last arrival on top publishes the barrier's epoch in
// gen, which every workgroup polls. attn/head count the arrivals of the
// attention splits of a KV head and of the head workgroups; within one
// persistent launch they only grow (the last arrival is recognised from the
// number of arrivals expected so far), one kernel per operation resets them.
// (The persistent kernel merges attention splits without a counter.)
struct Counters {
  uint32_t group[kBarGroups][64];
  uint32_t top[64];
  uint32_t gen[64];
  uint32_t attn[64][64];    // per (KV head, query-head pair), one kernel per operation
  uint32_t head[64];
};

struct DevParams {
  // shapes
  int L, H, A, K, D, F, V, G;   // G = A / K
  int qkv_rows;                 // (A + 2K) * D
  float eps;
  float attn_scale;             // 1/sqrt(D)
  float tau;
  int conf_measure;             // gate confidence: 0 max-prob, 1 top-2 margin, 2 negative entropy
  int exit_layer;               // 0 = ungated
  int page_size, page_shift;
  // weights
  const void* embed;            // [V][H]
  const LayerW* layers;         // [L] (device array)
  const float* g_final;         // [H]
  const void* ro_w;             // readout at exit_layer [H][H] (null if ungated)
  const float* ro_b;            // [H]
  // KV cache: pool[layer][page][kv_head][slot][D]
  void* kpool;
  void* vpool;
  int64_t layer_stride;         // elements per layer
  const int32_t* block_table;   // logical page -> physical page
  int32_t* hist_tok;            // [max_seq] input token of every position (written by layer 0)
  const float* rope_cos;        // [max_seq][D/2]
  const float* rope_sin;
  // Activations passed between phases, as tagged words: low 32 bits the fp32
  // value, high 32 bits the tag of the phase that wrote it (one 8-byte store).
  uint64_t* h;                  // [H] residual stream
  uint64_t* h_exit;             // [kMaxPending][H] residual stream at the exit layer (slot 0 unless lazy)
  uint64_t* z;                  // [H] readout output
  uint64_t* q;                  // [A*D]
  uint64_t* o;                  // [A*D]
  uint64_t* a;                  // [F]
  uint64_t* kvnew;              // [2*K*D] this step's K row, then V row (storage-rounded)
  uint64_t* dec;                // [5] exited, token, readout confidence, gate decision, readout token
  uint64_t* tw_all;             // all of the above, one block of tw_words words
  int64_t tw_words;
  uint64_t* attn_part;          // tagged attention partials [K][(G+1)/2][max_splits][2D + 4]
  int max_splits;
  float* head_part;             // [max_parts][kStatFloats]
  int max_parts;
  Counters* counters;
  StepCtl* ctl;
  // per-call ring (device arrays of n)
  int32_t* ring_tok;
  int32_t* ring_exit;
  int32_t* ring_would;          // may be null
  float* ring_conf;
  float* ring_mass;             // full-head mass ahead of the readout token (when nucleus)
  int nucleus;                  // the final head also measures the readout token's nucleus rank
  int lazy_fill;                // persistent kernel: > 1 = lazy fill with that many pending slots
  const int32_t* force_tok;     // may be null
  const int32_t* force_exit;    // may be null
  // debug outputs (device, may be null; only meaningful for single steps)
  float* dbg_logits_r;
  float* dbg_logits_f;
  float* dbg_h_final;
  // diagnostic timeline of the persistent kernel (may be null): workgroup 0
  // records the wall clock for phase e of the launch: [2e] when its inputs
  // are in LDS, [2e+1] when it has issued its outputs
  uint64_t* timeline;
  int timeline_cap;  // entries
};

// Buffers of the batched full-depth pass (ee_batched.hip), owned by the
// context and sized for chunks of at most max_positions positions.
struct BatchBuffers {
  int max_positions;
  float* X;               // [max_positions][H] residual stream
  float* Q;               // [max_positions][A*D] queries after RoPE
  float* O;               // [max_positions][A*D] attention output
  float* Act;             // [max_positions][F] SiLU(gate) * up
  float* gemm_ws;         // split-K partial sums
  size_t gemm_ws_floats;
  uint32_t* tile_ctr;     // arrivals per output tile (zero between launches)
  size_t n_tile_ctr;
  float* attn_ws;         // attention partial records of key splits
  size_t attn_ws_floats;
};

struct BatchPass {
  DevParams p;            // shapes, embedding, cache, RoPE tables, block table, token history, step record
  const LayerW* layers;   // host array [L] of the layers' device pointers
  BatchBuffers buf;
  int wbf16;
  int n_cu;
};

// Full depth over positions pos0 .. pos0 + n - 1 with input tokens d_tokens
// (device), in chunks of buf.max_positions: every layer's cache entries of
// those positions; the residual stream of the last chunk stays in buf.X.
hipError_t launch_batched_pass(const BatchPass& bp, int pos0, const int32_t* d_tokens, int n, hipStream_t s);
// tile counters the pass needs for chunks of max_positions and outputs of at most N_max rows
size_t batch_tile_counters(int max_positions, int N_max);

// Host launchers (defined in ee_kernels.hip).
hipError_t launch_decode_per_op(const DevParams& p, int wbf16, int pos0, int n, int head_wgs,
                                hipStream_t s);
// One persistent launch: the parameter block (pinned host memory) is copied
// into constant-memory slot `slot` on `stream` before the kernel starts.
struct PersistentLaunch {
  const DevParams* params_host;
  int slot;
  int wbf16;
  int nwg;
  size_t lds;
  hipStream_t stream;
};
hipError_t launch_decode_persistent(const PersistentLaunch& L, int pos0, int n);
hipError_t launch_prefill_per_op(const DevParams& p, int wbf16, int pos0, const int32_t* d_tokens,
                                 int n, int head_wgs, hipStream_t s);
hipError_t launch_prefill_persistent(const PersistentLaunch& L, int pos0, int n);
hipError_t launch_head_eval(const DevParams& p, int wbf16, const float* d_x, int readout,
                            int head_wgs, hipStream_t s);
// clear the per-call fields of the step record (all but next_token)
hipError_t launch_clear_step(StepCtl* c, hipStream_t s);
// copy the fp32 values of n tagged words to dst (device)
hipError_t launch_untag(float* dst, const uint64_t* src, int n, hipStream_t s);
// Device address of the library-resident scratch array (kScratchBytes) on
// `device`, which must be the current device; looked up once per device.
hipError_t scratch_address(int device, void** out);
size_t lds_bytes(const DevParams& p);
int fill_batch_slots(const DevParams& p);  // exit-layer states one lazy fill can batch
int chunks_per_lane(const DevParams& p, int wbf16);
int persistent_max_wgs_per_cu(const DevParams& p, int wbf16, size_t lds);

}  // namespace ee
