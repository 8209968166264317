/*
 * ee.h - C ABI of the gated early-exit decode library for MI355X (gfx950).
 *
 * One batch-1 decode step (the method of "One Size Does Not Fit All: Setting
 * Inference Depth from the Questions a Deployment Actually Asks", Section 4,
 * step five) runs the decoder layers up to an exit layer L_e, applies the
 * readout (a square matrix plus an offset whose result passes through the
 * model's own final RMSNorm and tied unembedding; Section 2 "Readout, or
 * lens", Appendix B), tests the readout's softmax max-probability against a
 * threshold tau (Section 2 "Confidence gate"), and then either emits the
 * readout's token, supplying the skipped layers' key/value cache entries by
 * projecting the exit-layer state through those layers' key and value
 * matrices (Section 4, step five), or runs the remaining layers and emits the
 * full model's token. Decoding is greedy.
 *
 * Conventions shared by every entry point
 *   - Return value: EE_OK (0) on success, a negative EE_E* code otherwise.
 *     ee_last_error() then describes the failure. No C++ exception crosses
 *     the ABI. After an error the context remains valid; ee_reset() restores
 *     a clean sequence state.
 *   - Host pointers are plain CPU memory owned by the caller. Device pointers
 *     (where an argument says so) are HIP device memory on the context's
 *     device, owned by the caller.
 *   - The library owns everything it allocates (repacked weights, KV pages,
 *     workspace) and frees it in ee_destroy().
 *   - A context is bound to one HIP stream and is not thread-safe.
 *   - exit_layer counts the decoder layers run before the readout, 1..L. The
 *     value 0 selects the plain ungated model (no readout, no gate): the
 *     baseline.
 *   - The gate exits iff conf > tau, compared in fp32. tau = +inf never exits;
 *     under the default measure tau <= 0 always exits (conf >= 1/V > 0).
 *     tau = NaN is EE_EINVAL.
 *   - conf is the readout's confidence under the selected measure (its max
 *     softmax probability unless ee_set_confidence_measure chose another),
 *     also on fallback steps; for the ungated model it is the full head's.
 *   - Argmax ties go to the lowest token id.
 */
#ifndef EE_H
#define EE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  EE_OK = 0,
  EE_EINVAL = -1,    /* bad argument: shape, name, size, exit layer without readout, NaN tau */
  EE_ESTATE = -2,    /* call not valid in this state (weights missing, decode before prefill) */
  EE_ENOMEM = -3,    /* device or host allocation failed */
  EE_EHIP = -4,      /* HIP runtime error */
  EE_ECAPACITY = -5, /* KV cache capacity (max_seq) would be exceeded */
  EE_EDEVICE = -6    /* the device reported an error (bounded wait timed out, bad token) */
};

enum { EE_F32 = 0, EE_BF16 = 1 }; /* storage type of matrices and KV cache */

enum {
  EE_CAL_EXIT_RATE = 0, /* tau so that a replay exits round(target*n) of n tokens */
  EE_CAL_MEDIAN = 1,    /* tau = median readout confidence (target ignored) */
  EE_CAL_NUCLEUS = 2    /* the paper's rule: lowest grid tau whose early answers are
                           acceptable (inside the full model's 0.9 nucleus) at least
                           a fraction target of the time */
};

/* When the KV-absence fill of an exited token runs (Section 4 step five). */
enum {
  EE_FILL_EAGER = 0, /* in the exit step itself (the default) */
  EE_FILL_LAZY = 1   /* deferred and batched: see ee_set_fill_policy */
};

/* Confidence measures the gate can compare with tau (Section 10 compares
 * these three softmax measures of the readout's distribution p). */
enum {
  EE_CONF_MAXPROB = 0,   /* p of the best token (the default; Section 2) */
  EE_CONF_MARGIN = 1,    /* best minus second-best probability, in [0, 1) */
  EE_CONF_NEGENTROPY = 2 /* sum_i p_i log p_i (natural log), in [-log V, 0] */
};

typedef struct ee_config {
  int32_t n_layers;   /* L */
  int32_t hidden;     /* H, multiple of 8 */
  int32_t n_q_heads;  /* A */
  int32_t n_kv_heads; /* K, A % K == 0, A/K <= 8 */
  int32_t head_dim;   /* D: a KV row of D elements is 128 or 256 bytes
                         (bf16: D = 64 or 128; fp32: D = 32 or 64) */
  int32_t ffn;        /* F, multiple of 8 */
  int32_t vocab;      /* V */
  float rope_base;    /* rotate-half RoPE base */
  float rms_eps;      /* RMSNorm epsilon */
  int32_t wdtype;     /* EE_F32 or EE_BF16 */
  int32_t max_seq;    /* KV capacity in positions */
  int32_t page_size;  /* positions per KV page, power of two */
} ee_config;

/* One named weight tensor. Matrices are canonical [out, in] row-major in the
 * configured storage type (fp32, or bf16 bit patterns); gains and offsets are
 * always fp32. ptr is host memory unless on_device != 0. Names:
 *   embed [V,H]; layers.{l}.attn_norm [H]; layers.{l}.wq [A*D,H];
 *   layers.{l}.wk [K*D,H]; layers.{l}.wv [K*D,H]; layers.{l}.wo [H,A*D];
 *   layers.{l}.mlp_norm [H]; layers.{l}.w_gate [F,H]; layers.{l}.w_up [F,H];
 *   layers.{l}.w_down [H,F]; final_norm [H]; readout.{L_e}.w [H,H];
 *   readout.{L_e}.b [H]   (l is 0-based, L_e is 1..L). */
typedef struct ee_tensor {
  const char* name;
  const void* ptr;
  int64_t nbytes;
  int32_t on_device;
} ee_tensor;

/* Per-step debug record filled by ee_decode_step_ex. Array pointers are host
 * memory and may be NULL; arrays a step does not produce are left untouched
 * (h_final and logits_full on exited steps, readout fields when ungated). */
typedef struct ee_debug {
  float* h_exit;          /* [H] residual stream after layer L_e */
  float* h_final;         /* [H] residual stream after layer L */
  float* logits_readout;  /* [V] readout logits */
  float* logits_full;     /* [V] full-head logits */
  int32_t token;          /* emitted token */
  int32_t exited;         /* branch taken */
  int32_t would_exit;     /* gate decision (conf > tau) before forcing */
  int32_t readout_token;  /* readout argmax, -1 when ungated */
  int32_t full_token;     /* full-head argmax, -1 when the upper layers were skipped */
  float conf;             /* readout confidence, selected measure (full head's when ungated) */
  float conf_full;        /* full head confidence, selected measure; NaN when skipped */
  float nucleus_mass;     /* full-head probability ahead of readout_token (order: probability
                             desc, id asc); readout_token is inside the 0.9 nucleus iff this
                             is < 0.9. NaN when skipped or ungated */
} ee_debug;

typedef struct ee_ctx ee_ctx;

/* Create a context on the current HIP device. hip_stream is a hipStream_t
 * (for instance torch's current stream) or NULL for a library-owned stream.
 * Allocates the KV pool for max_seq positions and the workspace.
 * Errors: EE_EINVAL (shape constraints above), EE_ENOMEM, EE_EHIP. */
int ee_create(const ee_config* cfg, void* hip_stream, ee_ctx** out);

/* Copy (and repack for the kernels' layouts) weights into library memory.
 * May be called several times; a later tensor of the same name replaces the
 * earlier one. Decoding needs every non-readout tensor; gated decoding at
 * exit layer L_e also needs readout.{L_e}.w and .b. Synchronous.
 * Errors: EE_EINVAL (unknown name, wrong nbytes), EE_ENOMEM, EE_EHIP. */
int ee_load_weights(ee_ctx* ctx, const ee_tensor* tensors, int32_t n_tensors);

/* Prompt pass at full depth, ungated, over positions pos..pos+n-1 (host token
 * ids in [0,V)). The gate of Section 4 step five applies to produced tokens;
 * a prompt runs through the unmodified model, as the prompts of Section 4
 * step one do, so every layer's cache entries of the prompt are exact.
 * Writes every layer's KV entries and returns in
 * *out_first_token the full head's argmax at the last prompt position, which
 * becomes the next decode step's input. Synchronous.
 * Errors: EE_ESTATE (weights incomplete), EE_EINVAL (n <= 0, bad token),
 * EE_ECAPACITY, EE_EHIP, EE_EDEVICE. */
int ee_prefill(ee_ctx* ctx, const int32_t* tokens, int32_t n, int32_t* out_first_token);

/* One gated decode step on the last emitted token; syncs once.
 * Outputs (host, any may be NULL): emitted token, exited flag, conf.
 * Errors: EE_ESTATE (no prefill yet / weights incomplete), EE_EINVAL
 * (exit_layer out of 0..L or without a loaded readout, NaN tau),
 * EE_ECAPACITY, EE_EHIP, EE_EDEVICE. */
int ee_decode_step(ee_ctx* ctx, float tau, int32_t exit_layer,
                   int32_t* out_token, int32_t* out_exited, float* out_conf);

/* n gated decode steps enqueued as one device program; each step's input is
 * the previous step's output token, read on the device, so the host never
 * waits per token. One sync at the end. tokens/exited/conf are host arrays of
 * n entries (any may be NULL). Errors as ee_decode_step, plus EE_EINVAL for
 * n <= 0. */
int ee_decode_n(ee_ctx* ctx, float tau, int32_t exit_layer, int32_t n,
                int32_t* tokens, int32_t* exited, float* conf);

/* ee_decode_n for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * it calls no hipMalloc, hipFree or other allocating routine. The outputs
 * go to caller-owned device arrays of n entries on the context's device
 * (d_tokens, d_exited as 0/1, d_conf; none may be NULL), and the call's
 * working set (tagged activation words, attention and head partial records,
 * barrier counters) lives in a library-resident scratch array of 4 MiB per
 * device, held until the process ends, instead of the context's own
 * buffers. The scratch is cleared at the start of every call. All calls on
 * one device share that device's scratch: calls that overlap in time on one
 * device (several contexts on different streams) race, and the caller must
 * order them. One sync at the end, as ee_decode_n; the results equal
 * ee_decode_n's. Errors as ee_decode_n, plus EE_EINVAL for a NULL output
 * and EE_ECAPACITY when the context's working set (it grows with max_seq
 * through the attention partial records) exceeds the scratch. */
int ee_decode_n_noalloc(ee_ctx* ctx, float tau, int32_t exit_layer, int32_t n,
                        int32_t* d_tokens, int32_t* d_exited, float* d_conf);

/* ee_decode_n with optional imposed inputs (host arrays of n, may be NULL):
 * force_tokens[i] replaces step i's input token (teacher forcing; the first
 * step may then run without a prior prefill output), force_exit[i] is -1
 * (use the gate), 0 (never exit) or 1 (always exit); imposed exit decisions
 * are the paper's timing method (Appendix C). would_exit[i] receives the gate's
 * own decision. Errors as ee_decode_n, plus EE_EINVAL for bad forced values. */
int ee_decode_n_ex(ee_ctx* ctx, float tau, int32_t exit_layer, int32_t n,
                   const int32_t* force_tokens, const int32_t* force_exit,
                   int32_t* tokens, int32_t* exited, float* conf, int32_t* would_exit);

/* One step with an optional input token (-1 = last emitted), an optional
 * imposed branch (-1 gate, 0 never exit, 1 always exit) and a debug record
 * (may be NULL). Test hook; runs the same device program as ee_decode_n. */
int ee_decode_step_ex(ee_ctx* ctx, float tau, int32_t exit_layer, int32_t input_token,
                      int32_t force_exit, ee_debug* dbg);

/* Calibrate tau on the device (Section 4, step four): for each prompt,
 * reset, prefill, then n_gen steps at tau = +inf (full depth, readout
 * computed), recording the readout confidences. EE_CAL_EXIT_RATE: with the n
 * recorded values sorted ascending c_1..c_n and k = floor(target*n + 1/2),
 * tau = c_(n-k) (+inf for k = 0, -inf for k = n). EE_CAL_MEDIAN: the median.
 * EE_CAL_NUCLEUS (Section 4 step four, Section 2 "Nucleus"): the final head
 * also measures, per step, the full model's probability mass ahead of the
 * readout's token; the token is acceptable iff that mass is below 0.9. tau is
 * the smallest of 0.00, 0.01, ..., 0.99 for which the steps with confidence
 * above tau are non-empty and acceptable with frequency >= target (the paper
 * uses 0.9); +inf when none qualifies.
 * prompts holds the prompts back to back (host), prompt_lens their lengths.
 * Leaves the context reset. Errors: EE_EINVAL, EE_ESTATE, EE_ECAPACITY,
 * EE_EHIP, EE_EDEVICE. */
int ee_calibrate_threshold(ee_ctx* ctx, const int32_t* prompts, const int32_t* prompt_lens,
                           int32_t n_prompts, int32_t n_gen, int32_t exit_layer,
                           int32_t mode, float target, float* out_tau);

/* The per-step record of the most recent ee_calibrate_threshold call on ctx
 * (test hook): confs[i] the readout confidence of recorded step i (prompt by
 * prompt, n_gen steps each, in order) and, for EE_CAL_NUCLEUS, masses[i] the
 * full model's probability mass ahead of the readout's token (the token is
 * acceptable iff it is below 0.9; Section 4 step four); NaN for the other
 * modes. Host arrays of n entries, either may be NULL.
 * Errors: EE_ESTATE (no calibration yet), EE_EINVAL (n is not the number of
 * recorded steps). */
int ee_calibration_record(ee_ctx* ctx, int32_t n, float* confs, float* masses);

/* Periodic full-depth refresh (Section 11): recompute the cache entries of
 * the n most recent positions at every layer from their own input tokens,
 * replacing the entries projected for exited tokens by the KV-absence fill.
 * Runs the full-depth pass of the prompt over those positions, batched (see
 * ee_set_prefill_chunk): every weight is read once for all n positions. The
 * position and the next input token are unchanged. Errors: EE_EINVAL (n outside
 * 1..position), EE_ESTATE, EE_EHIP, EE_EDEVICE. */
int ee_refresh(ee_ctx* ctx, int32_t n);

/* How full-depth passes over many positions run (ee_prefill, ee_refresh):
 * positions > 0 batches chunks of at most that many positions (capped at
 * 1024, and the default) through each layer together, so every weight is
 * read once per chunk: per layer a tiled matrix product for the query, key
 * and value projections (with RoPE and the cache stores), causal attention
 * of the chunk's queries over every cached position up to their own, and
 * matrix products for the output projection and the feed-forward block.
 * 0 runs one position per step through the decode program (the earlier
 * path; kept as a cross-check). Results agree to rounding (the summation
 * order differs). Errors: EE_EINVAL (positions < 0). */
int ee_set_prefill_chunk(ee_ctx* ctx, int32_t positions);

/* EE_FILL_LAZY: in the persistent program an exit step only keeps its
 * exit-layer state; the cache entries of consecutive exited tokens are
 * written together (each skipped layer's W_k/W_v rows read once per batch)
 * before the next step that runs the upper layers, when the batch is full
 * (up to 8 tokens, fewer for wide models) and before the call returns, so
 * the cache is complete whenever a call has returned. The entries are
 * bit-identical to the eager fill's. The one-kernel-per-operation program
 * always fills eagerly. Errors: EE_EINVAL (unknown policy). */
int ee_set_fill_policy(ee_ctx* ctx, int32_t policy);

/* Select the confidence measure (EE_CONF_*) for the gate (exit iff the
 * measure exceeds tau), for the conf values decode calls report, for
 * calibration and for ee_head_eval. All three come from the same single pass
 * over the vocabulary. Takes effect at the next call; the context starts with
 * EE_CONF_MAXPROB. Errors: EE_EINVAL (unknown measure). */
int ee_set_confidence_measure(ee_ctx* ctx, int32_t measure);

/* Replace the offset b (H fp32) of the readout at exit_layer: the offset of
 * the readout's affine map (Section 4 step two, Appendix B). Asynchronously
 * on the context's stream (no sync): later steps enqueued on the stream see
 * it. Errors: EE_EINVAL (no readout at that layer), EE_EHIP. */
int ee_set_readout_bias(ee_ctx* ctx, int32_t exit_layer, const float* b, int32_t on_device);

/* Evaluate one head on a caller vector x (H fp32, host): layer 0 = the full
 * head (final RMSNorm + unembedding), layer L_e = the readout at L_e followed
 * by the full head. Runs the decode step's head kernel. Outputs (any may be
 * NULL): argmax token, confidence under the selected measure, logits [V]
 * (host). Test hook. */
int ee_head_eval(ee_ctx* ctx, int32_t readout_layer, const float* x,
                 int32_t* out_token, float* out_conf, float* out_logits);

/* Copy the cache entries of (layer, position) as fp32 into k_out and v_out
 * (host, K*D each, [kv_head][d], post-RoPE keys). Test hook.
 * Errors: EE_EINVAL (layer or pos out of range / not yet written). */
int ee_read_kv(ee_ctx* ctx, int32_t layer, int32_t pos, float* k_out, float* v_out);

/* Select the device program used for decoding and prefill: wgs_per_cu >= 1
 * runs one persistent cooperative kernel per call with that many workgroups
 * per compute unit; a negative value selects as many as can be co-resident
 * (the default); 0 runs one kernel per operation.
 * Errors: EE_EINVAL (more workgroups than can be co-resident). */
int ee_set_persistent(ee_ctx* ctx, int32_t wgs_per_cu);

/* Run the persistent program with exactly nwg workgroups in total. Every
 * phase distributes its work over any grid size, so results equal those of
 * the default grid (up to the summation order of the head's exp-sums); a grid
 * smaller than the number of compute units leaves units idle.
 * Errors: EE_EINVAL (nwg < 1 or more than can be co-resident),
 * EE_ESTATE (no persistent-kernel parameter slot). */
int ee_set_persistent_grid(ee_ctx* ctx, int32_t nwg);

/* Diagnostic timeline of the persistent kernel (test hook): with capacity > 0,
 * later launches record the device wall clock (hipDeviceAttributeWallClockRate
 * ticks) in workgroup 0 around every phase of the launch — entry 2e when phase
 * e (1-based: the phases of each step in order, five per layer, then the
 * readout, its head, and the KV fill or the final head) has requested its
 * weights and is about to wait for its input, 2e+1 when it has issued its
 * outputs — up to capacity entries. capacity 0 turns it off.
 * ee_read_timeline copies the first n entries of the latest launch into out
 * (host). */
int ee_set_timeline(ee_ctx* ctx, int32_t capacity);
int ee_read_timeline(ee_ctx* ctx, uint64_t* out, int32_t n);

/* Streaming-read ceiling of the device: a plain kernel reads `bytes` (rounded
 * down to 16-byte words) of a buffer the call allocates and frees, with
 * 16-byte coalesced loads, each workgroup (eight per compute unit) streaming
 * one contiguous range; one warm-up launch, then
 * `reps` timed launches on the context's stream (HIP events). *out_gbps =
 * bytes / median launch time, in 1e9 B/s. The decode path's achieved bandwidth
 * is reported against this ceiling as well as against the spec-sheet peak.
 * Measurement tool, not part of decoding.
 * Errors: EE_EINVAL (bytes < 16, reps < 1, out_gbps NULL), EE_ENOMEM,
 * EE_EHIP. */
int ee_stream_probe(ee_ctx* ctx, int64_t bytes, int32_t reps, float* out_gbps);

/* Device time in milliseconds of the most recent ee_decode_n/_ex call's
 * kernels, measured with HIP events on the context's stream. */
int ee_last_decode_ms(ee_ctx* ctx, float* out_ms);

/* Sequence position (number of cached positions). */
int32_t ee_position(const ee_ctx* ctx);

/* Drop the KV cache contents and position, keep weights. */
int ee_reset(ee_ctx* ctx);

/* Message of the most recent error on ctx (empty string if none). With
 * ctx == NULL: the message of this thread's most recent ee_create failure. */
const char* ee_last_error(const ee_ctx* ctx);

void ee_destroy(ee_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* EE_H */
