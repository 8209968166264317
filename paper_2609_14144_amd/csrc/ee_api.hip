// C ABI of the gated early-exit decode library: context, weight loading and
// repacking, paged KV allocation, step launching, calibration, test hooks.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <initializer_list>
#include <atomic>
#include <map>
#include <new>
#include <random>
#include <set>
#include <stdexcept>
#include <string>
#include <vector>

#include "ee.h"
#include "ee_internal.h"

using ee::DevParams;

namespace ee {
hipError_t launch_stream_read(const void* p, int64_t n, int n_cu, uint32_t* sink, hipStream_t s);  // ee_probe.hip
}

struct ee_ctx {
  ee_config cfg{};
  int wbf16 = 0;
  size_t esz = 4;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  int device = 0;
  int n_cu = 0;

  void* embed = nullptr;
  std::vector<void*> wqkv, wo, wgu, wd;
  std::vector<float*> g_attn, g_mlp;
  float* g_final = nullptr;
  std::map<int, std::pair<void*, float*>> readout;
  ee::LayerW* d_layers = nullptr;
  std::vector<ee::LayerW> h_layers;   // the same pointers, host side (batched pass)
  ee::BatchBuffers bbuf{};            // batched full-depth pass (prompt, refresh)
  int prefill_chunk = -1;             // -1: batched in chunks of bbuf.max_positions; 0: one position per step

  void* kpool = nullptr;
  void* vpool = nullptr;
  int64_t layer_stride = 0;
  int n_pages = 0;
  int32_t* d_block_table = nullptr;
  int32_t* d_hist = nullptr;         // input token of every position
  int32_t* h_block_table = nullptr;  // pinned
  int pages_mapped = 0;
  std::vector<int32_t> free_pages;

  float* d_cos = nullptr;
  float* d_sin = nullptr;
  // tagged activation words (value + producer tag), one block
  uint64_t* d_tw = nullptr;
  int64_t tw_words = 0;
  uint64_t *d_h = nullptr, *d_hexit = nullptr, *d_z = nullptr, *d_q = nullptr, *d_o = nullptr,
           *d_a = nullptr, *d_kvnew = nullptr, *d_dec = nullptr;
  uint64_t* d_attn_part = nullptr;  // tagged, inside d_tw
  int max_splits = 0;
  float* d_head_part = nullptr;
  int max_parts = 0;
  ee::Counters* d_counters = nullptr;
  ee::StepCtl* d_ctl = nullptr;

  int ring_cap = 0;
  int32_t *d_ring_tok = nullptr, *d_ring_exit = nullptr, *d_ring_would = nullptr;
  float* d_ring_conf = nullptr;
  float* d_ring_mass = nullptr;
  std::vector<float> cal_confs, cal_masses;  // record of the latest calibration (test hook)
  bool fill_lazy = false;  // persistent program: batch the KV fill of consecutive exits
  int fill_slots = 0;      // exit-layer states one batched fill can take
  bool nucleus = false;   // steps also measure the readout token's nucleus rank (calibration, debug)
  int force_cap = 0;
  int32_t *d_force_tok = nullptr, *d_force_exit = nullptr;
  float *d_dbg_r = nullptr, *d_dbg_f = nullptr, *d_x = nullptr;

  std::set<std::string> loaded;
  int pos = 0;
  bool have_next = false;
  bool persistent = true;
  int head_wgs = 0;
  int nwg_persistent = 0;
  int max_wgs_per_cu = 0;
  int conf_measure = EE_CONF_MAXPROB;
  size_t lds = 0;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  float last_ms = 0.f;
  int slot = -1;                       // constant-memory parameter slot (persistent kernel)
  uint64_t* d_timeline = nullptr;
  int timeline_cap = 0;
  DevParams* params_pinned = nullptr;  // staging of the parameter block
  void* scratch = nullptr;             // this device's library-resident scratch (ee_decode_n_noalloc)
  std::string err;
};

namespace {

// Section 2's nucleus: the smallest set of most probable tokens holding 0.9
// of the full model's probability.
constexpr float kNucleusTopP = 0.9f;

thread_local std::string g_create_err;  // last ee_create failure (no context exists)
std::atomic<uint32_t> g_slots{0};       // parameter slots in use (one bit each)

int take_slot() {
  uint32_t cur = g_slots.load();
  while (true) {
    int i = 0;
    while (i < ee::kParamSlots && (cur >> i & 1u)) ++i;
    if (i == ee::kParamSlots) return -1;
    if (g_slots.compare_exchange_weak(cur, cur | (1u << i))) return i;
  }
}

void give_slot(int i) {
  if (i >= 0) g_slots.fetch_and(~(1u << i));
}

int fail(ee_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg;
  return code;
}

// Record a message for an exception caught at the ABI (never throws: a
// failed assignment leaves the message empty).
void note_exception(ee_ctx* c, const char* msg) noexcept {
  try {
    if (c) c->err = msg;
    else g_create_err = msg;
  } catch (...) {
    if (c) c->err.clear();
    else g_create_err.clear();
  }
}

template <typename F>
int guarded(ee_ctx* c, F&& f) noexcept {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    note_exception(c, "out of host memory");
    return EE_ENOMEM;
  } catch (const std::length_error&) {
    note_exception(c, "out of host memory (size limit)");
    return EE_ENOMEM;
  } catch (...) {
    note_exception(c, "unexpected C++ exception inside the library");
    return EE_EINVAL;
  }
}

int hip_fail(ee_ctx* c, hipError_t e, const char* what) {
  return fail(c, EE_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIPCHK(ctx, call)                                     \
  do {                                                        \
    hipError_t e_ = (call);                                   \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #call);  \
  } while (0)

template <typename T>
int dalloc(ee_ctx* c, T** p, size_t bytes) {
  void* q = nullptr;
  if (hipMalloc(&q, bytes ? bytes : 16) != hipSuccess) {
    (void)hipGetLastError();
    return fail(c, EE_ENOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
  }
  const hipError_t e = hipMemset(q, 0, bytes ? bytes : 16);
  if (e != hipSuccess) {
    (void)hipFree(q);
    return hip_fail(c, e, "hipMemset");
  }
  *p = static_cast<T*>(q);
  return EE_OK;
}

void dfree(void* p) {
  if (p) (void)hipFree(p);
}

int elems_per_chunk(const ee_ctx* c) { return c->wbf16 ? 8 : 4; }

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

int validate_config(const ee_config* g, std::string& why) {
  const int N = g->wdtype == EE_BF16 ? 8 : 4;
  if (g->wdtype != EE_F32 && g->wdtype != EE_BF16) { why = "wdtype must be EE_F32 or EE_BF16"; return 0; }
  if (g->n_layers < 1 || g->n_layers > 512) { why = "n_layers out of range"; return 0; }
  if (g->hidden < 8 || g->hidden % 8) { why = "hidden must be a positive multiple of 8"; return 0; }
  if (g->ffn < 8 || g->ffn % 8) { why = "ffn must be a positive multiple of 8"; return 0; }
  if (g->n_kv_heads < 1 || g->n_kv_heads > 16) { why = "n_kv_heads must be 1..16"; return 0; }
  if (g->n_q_heads < 1 || g->n_q_heads % g->n_kv_heads) { why = "n_q_heads must be a multiple of n_kv_heads"; return 0; }
  if (g->n_q_heads / g->n_kv_heads > ee::kMaxGroup) { why = "more than 8 query heads per kv head"; return 0; }
  if (g->head_dim < 2 || g->head_dim > ee::kMaxHeadDim || g->head_dim % N) {
    why = "head_dim must be a multiple of 16 bytes of storage and at most 256"; return 0;
  }
  if (64 % (g->head_dim / N)) { why = "head_dim / elems-per-16-bytes must divide 64"; return 0; }
  if ((g->head_dim * (g->wdtype == EE_BF16 ? 2 : 4)) % 128) {
    why = "a KV row (head_dim elements) must fill whole 128-byte lines"; return 0;
  }
  if (g->head_dim * (g->wdtype == EE_BF16 ? 2 : 4) > 256) {
    why = "a KV row (head_dim elements) must be at most 256 bytes"; return 0;
  }
  if (g->vocab < 2) { why = "vocab must be >= 2"; return 0; }
  if (g->max_seq < 1) { why = "max_seq must be >= 1"; return 0; }
  if (!is_pow2(g->page_size)) { why = "page_size must be a power of two"; return 0; }
  if (!(g->rms_eps > 0.f) || !(g->rope_base > 0.f)) { why = "rms_eps and rope_base must be positive"; return 0; }
  return 1;
}

// The tagged activation words of a decode call, in one block: h, h_exit
// (kMaxPending slots), z, q, o, a, this step's K/V row, the gate record and
// the attention partial records, each part starting on a 256-byte boundary.
constexpr int kTwParts = 9;
int64_t tw_layout(const ee_config& g, int64_t off[kTwParts]) {
  const int64_t H = g.hidden, A = g.n_q_heads, K = g.n_kv_heads, D = g.head_dim, F = g.ffn;
  const int64_t pairs = ((A / K) + 1) / 2;
  const int64_t splits = (g.max_seq + ee::kAttnSplit - 1) / ee::kAttnSplit;
  const int64_t sizes[kTwParts] = {H, int64_t(ee::kMaxPending) * H, H, A * D, A * D, F, 2 * K * D, 8,
                                   K * pairs * splits * (2 * D + 4)};
  int64_t total = 0;
  for (int i = 0; i < kTwParts; ++i) {
    off[i] = total;
    total += (sizes[i] + 31) & ~int64_t(31);
  }
  return total;
}

void tw_bind(uint64_t* base, const int64_t off[kTwParts], uint64_t** const ptrs[kTwParts]) {
  for (int i = 0; i < kTwParts; ++i) *ptrs[i] = base + off[i];
}

DevParams make_params(const ee_ctx* c, float tau, int exit_layer) {
  const ee_config& g = c->cfg;
  DevParams p{};
  p.L = g.n_layers; p.H = g.hidden; p.A = g.n_q_heads; p.K = g.n_kv_heads; p.D = g.head_dim;
  p.F = g.ffn; p.V = g.vocab; p.G = g.n_q_heads / g.n_kv_heads;
  p.qkv_rows = (p.A + 2 * p.K) * p.D;
  p.eps = g.rms_eps;
  p.attn_scale = static_cast<float>(1.0 / sqrt(static_cast<double>(p.D)));
  p.tau = tau;
  p.conf_measure = c->conf_measure;
  p.exit_layer = exit_layer;
  p.page_size = g.page_size;
  int sh = 0;
  while ((1 << sh) < g.page_size) ++sh;
  p.page_shift = sh;
  p.embed = c->embed;
  p.layers = c->d_layers;
  p.g_final = c->g_final;
  if (exit_layer > 0) {
    auto it = c->readout.find(exit_layer);
    p.ro_w = it->second.first;
    p.ro_b = it->second.second;
  }
  p.kpool = c->kpool; p.vpool = c->vpool; p.layer_stride = c->layer_stride;
  p.block_table = c->d_block_table;
  p.hist_tok = c->d_hist;
  p.rope_cos = c->d_cos; p.rope_sin = c->d_sin;
  p.h = c->d_h; p.h_exit = c->d_hexit; p.z = c->d_z; p.q = c->d_q; p.o = c->d_o; p.a = c->d_a;
  p.kvnew = c->d_kvnew; p.dec = c->d_dec; p.tw_all = c->d_tw; p.tw_words = c->tw_words;
  p.attn_part = c->d_attn_part; p.max_splits = c->max_splits;
  p.head_part = c->d_head_part; p.max_parts = c->max_parts;
  p.counters = c->d_counters; p.ctl = c->d_ctl;
  p.timeline = c->d_timeline;
  p.timeline_cap = c->timeline_cap;
  return p;
}

int ensure_pages(ee_ctx* c, int pos_end) {
  if (pos_end > c->cfg.max_seq)
    return fail(c, EE_ECAPACITY, "KV capacity exceeded: need " + std::to_string(pos_end) +
                                     " positions, max_seq " + std::to_string(c->cfg.max_seq));
  const int need = (pos_end + c->cfg.page_size - 1) / c->cfg.page_size;
  const int first = c->pages_mapped;
  while (c->pages_mapped < need) {
    c->h_block_table[c->pages_mapped++] = c->free_pages.back();
    c->free_pages.pop_back();
  }
  if (c->pages_mapped > first)
    HIPCHK(c, hipMemcpyAsync(c->d_block_table + first, c->h_block_table + first,
                             sizeof(int32_t) * (c->pages_mapped - first), hipMemcpyHostToDevice,
                             c->stream));
  return EE_OK;
}

void reset_pages(ee_ctx* c) {
  c->pages_mapped = 0;
  c->free_pages.resize(c->n_pages);
  for (int i = 0; i < c->n_pages; ++i) c->free_pages[i] = i;
  // A fixed scrambled order: physical page order differs from logical order.
  std::mt19937 rng(12345u);
  std::shuffle(c->free_pages.begin(), c->free_pages.end(), rng);
}

int ensure_ring(ee_ctx* c, int n) {
  if (n <= c->ring_cap) return EE_OK;
  dfree(c->d_ring_tok); dfree(c->d_ring_exit); dfree(c->d_ring_would); dfree(c->d_ring_conf);
  dfree(c->d_ring_mass);
  c->d_ring_tok = c->d_ring_exit = c->d_ring_would = nullptr;
  c->d_ring_conf = c->d_ring_mass = nullptr;
  c->ring_cap = 0;
  int r;
  if ((r = dalloc(c, &c->d_ring_tok, sizeof(int32_t) * n))) return r;
  if ((r = dalloc(c, &c->d_ring_exit, sizeof(int32_t) * n))) return r;
  if ((r = dalloc(c, &c->d_ring_would, sizeof(int32_t) * n))) return r;
  if ((r = dalloc(c, &c->d_ring_conf, sizeof(float) * n))) return r;
  if ((r = dalloc(c, &c->d_ring_mass, sizeof(float) * n))) return r;
  c->ring_cap = n;
  return EE_OK;
}

int ensure_force(ee_ctx* c, int n) {
  if (n <= c->force_cap) return EE_OK;
  dfree(c->d_force_tok); dfree(c->d_force_exit);
  c->d_force_tok = c->d_force_exit = nullptr;
  c->force_cap = 0;
  int r;
  if ((r = dalloc(c, &c->d_force_tok, sizeof(int32_t) * n))) return r;
  if ((r = dalloc(c, &c->d_force_exit, sizeof(int32_t) * n))) return r;
  c->force_cap = n;
  return EE_OK;
}

bool weights_ready(const ee_ctx* c) {
  return c->loaded.size() >= static_cast<size_t>(2 + 9 * c->cfg.n_layers) &&
         c->loaded.count("embed") && c->loaded.count("final_norm");
}

int check_gate_args(ee_ctx* c, float tau, int exit_layer) {
  if (isnan(tau)) return fail(c, EE_EINVAL, "tau is NaN");
  if (exit_layer < 0 || exit_layer > c->cfg.n_layers)
    return fail(c, EE_EINVAL, "exit_layer must be in 0..n_layers");
  if (exit_layer > 0 && !c->readout.count(exit_layer))
    return fail(c, EE_EINVAL, "no readout loaded at layer " + std::to_string(exit_layer));
  if (!weights_ready(c)) return fail(c, EE_ESTATE, "weights not fully loaded");
  return EE_OK;
}

// Caller-owned device outputs of an allocation-free decode call; its working
// set is bound to the library-resident scratch.
struct NoAlloc {
  int32_t* tok;
  int32_t* exited;
  float* conf;
};

// Bytes of the scratch a decode call of this context uses: the tagged words,
// the head partial records and the barrier counters.
size_t scratch_need(const ee_ctx* c, int64_t off[kTwParts], size_t* head_off, size_t* ctr_off) {
  const int64_t words = tw_layout(c->cfg, off);
  size_t b = static_cast<size_t>(words) * 8;
  *head_off = b;
  b += (static_cast<size_t>(c->max_parts) * ee::kStatFloats * 4 + 255) & ~size_t(255);
  *ctr_off = b;
  return b + ((sizeof(ee::Counters) + 255) & ~size_t(255));
}

int bind_scratch(ee_ctx* c, DevParams& p) {
  int64_t off[kTwParts];
  size_t head_off, ctr_off;
  const size_t need = scratch_need(c, off, &head_off, &ctr_off);
  if (need > ee::kScratchBytes)
    return fail(c, EE_ECAPACITY, "this context's decode working set needs " + std::to_string(need) +
                                     " bytes of scratch; the library-resident scratch holds " +
                                     std::to_string(ee::kScratchBytes) + " (reduce max_seq)");
  char* base = static_cast<char*>(c->scratch);
  uint64_t** const ptrs[kTwParts] = {&p.h, &p.h_exit, &p.z, &p.q, &p.o, &p.a, &p.kvnew, &p.dec, &p.attn_part};
  tw_bind(reinterpret_cast<uint64_t*>(base), off, ptrs);
  p.tw_all = reinterpret_cast<uint64_t*>(base);
  p.tw_words = static_cast<int64_t>(head_off / 8);
  p.head_part = reinterpret_cast<float*>(base + head_off);
  p.counters = reinterpret_cast<ee::Counters*>(base + ctr_off);
  return EE_OK;
}

// Launch n steps (decode, or prompt positions when prefill) and wait. With
// na set, the outputs go to the caller's device arrays and the working set
// to the library-resident scratch: nothing is allocated.
int run_steps(ee_ctx* c, float tau, int exit_layer, int n, const int32_t* d_force_tok,
              const int32_t* d_force_exit, bool prefill, bool debug, const NoAlloc* na = nullptr) {
  int r;
  DevParams p = make_params(c, tau, prefill ? 0 : exit_layer);
  if (na && (r = bind_scratch(c, p))) return r;
  if (!na && (r = ensure_ring(c, n))) return r;
  if ((r = ensure_pages(c, c->pos + n))) return r;
  if (na) {
    p.ring_tok = na->tok; p.ring_exit = na->exited; p.ring_conf = na->conf;
    p.ring_would = nullptr; p.ring_mass = nullptr;
  } else {
    p.ring_tok = c->d_ring_tok; p.ring_exit = c->d_ring_exit;
    p.ring_would = c->d_ring_would; p.ring_conf = c->d_ring_conf;
    p.ring_mass = c->d_ring_mass;
  }
  p.nucleus = c->nucleus && !prefill;
  p.force_tok = d_force_tok;
  p.force_exit = d_force_exit;
  if (debug) {
    p.dbg_logits_r = c->d_dbg_r;
    p.dbg_logits_f = c->d_dbg_f;
  }
  // Clear the step record except next_token, the first step's input.
  if (na) {
    hipError_t ce = ee::launch_clear_step(c->d_ctl, c->stream);
    if (ce != hipSuccess) return hip_fail(c, ce, "step record clear");
  } else {
    HIPCHK(c, hipMemsetAsync(reinterpret_cast<char*>(c->d_ctl) + offsetof(ee::StepCtl, exited), 0,
                             offsetof(ee::StepCtl, pad) - offsetof(ee::StepCtl, exited), c->stream));
  }
  HIPCHK(c, hipEventRecord(c->ev0, c->stream));
  hipError_t e;
  const bool pers = c->persistent && c->nwg_persistent > 0 && c->slot >= 0;
  if (pers) {
    p.lazy_fill = (c->fill_lazy && c->fill_slots > 1) ? c->fill_slots : 0;
    *c->params_pinned = p;
    const ee::PersistentLaunch L{c->params_pinned, c->slot, c->wbf16, c->nwg_persistent, c->lds, c->stream};
    e = prefill ? ee::launch_prefill_persistent(L, c->pos, n) : ee::launch_decode_persistent(L, c->pos, n);
  } else if (prefill) {
    e = ee::launch_prefill_per_op(p, c->wbf16, c->pos, d_force_tok, n, c->head_wgs, c->stream);
  } else {
    e = ee::launch_decode_per_op(p, c->wbf16, c->pos, n, c->head_wgs, c->stream);
  }
  if (e != hipSuccess) return hip_fail(c, e, "kernel launch");
  HIPCHK(c, hipEventRecord(c->ev1, c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  HIPCHK(c, hipEventElapsedTime(&c->last_ms, c->ev0, c->ev1));
  ee::StepCtl ctl;
  HIPCHK(c, hipMemcpy(&ctl, c->d_ctl, sizeof(ctl), hipMemcpyDeviceToHost));
  if (ctl.error != ee::kErrNone || ctl.abort) {
    c->have_next = false;
    return fail(c, EE_EDEVICE, ctl.error == ee::kErrToken  ? "device: token id out of range"
                               : ctl.error == ee::kErrWait ? "device: bounded wait for a phase's input timed out"
                                                           : "device: bounded grid wait timed out");
  }
  c->pos += n;
  c->have_next = true;
  return EE_OK;
}

// fp32 values of n tagged device words into host memory
int copy_untag(ee_ctx* c, float* dst, const uint64_t* src, size_t n) {
  std::vector<uint64_t> w(n);
  HIPCHK(c, hipMemcpy(w.data(), src, n * 8, hipMemcpyDeviceToHost));
  for (size_t i = 0; i < n; ++i) {
    const uint32_t b = static_cast<uint32_t>(w[i]);
    memcpy(dst + i, &b, 4);
  }
  return EE_OK;
}

int copy_ring(ee_ctx* c, int n, int32_t* tokens, int32_t* exited, float* conf, int32_t* would) {
  if (tokens) HIPCHK(c, hipMemcpy(tokens, c->d_ring_tok, sizeof(int32_t) * n, hipMemcpyDeviceToHost));
  if (exited) HIPCHK(c, hipMemcpy(exited, c->d_ring_exit, sizeof(int32_t) * n, hipMemcpyDeviceToHost));
  if (conf) HIPCHK(c, hipMemcpy(conf, c->d_ring_conf, sizeof(float) * n, hipMemcpyDeviceToHost));
  if (would) HIPCHK(c, hipMemcpy(would, c->d_ring_would, sizeof(int32_t) * n, hipMemcpyDeviceToHost));
  return EE_OK;
}

int upload_force(ee_ctx* c, int n, const int32_t* force_tokens, const int32_t* force_exit) {
  int r;
  if (!force_tokens && !force_exit) return EE_OK;
  if ((r = ensure_force(c, n))) return r;
  if (force_tokens) {
    for (int i = 0; i < n; ++i)
      if (force_tokens[i] < 0 || force_tokens[i] >= c->cfg.vocab)
        return fail(c, EE_EINVAL, "force_tokens[" + std::to_string(i) + "] out of range");
    HIPCHK(c, hipMemcpy(c->d_force_tok, force_tokens, sizeof(int32_t) * n, hipMemcpyHostToDevice));
  }
  if (force_exit) {
    for (int i = 0; i < n; ++i)
      if (force_exit[i] < -1 || force_exit[i] > 1)
        return fail(c, EE_EINVAL, "force_exit values must be -1, 0 or 1");
    HIPCHK(c, hipMemcpy(c->d_force_exit, force_exit, sizeof(int32_t) * n, hipMemcpyHostToDevice));
  }
  return EE_OK;
}

int decode_common(ee_ctx* c, float tau, int exit_layer, int n, const int32_t* force_tokens,
                  const int32_t* force_exit, bool debug) {
  int r;
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (n <= 0) return fail(c, EE_EINVAL, "n must be positive");
  if ((r = check_gate_args(c, tau, exit_layer))) return r;
  if (!force_tokens && !c->have_next)
    return fail(c, EE_ESTATE, "no input token: run ee_prefill first (or force the input tokens)");
  if ((r = upload_force(c, n, force_tokens, force_exit))) return r;
  return run_steps(c, tau, exit_layer, n, force_tokens ? c->d_force_tok : nullptr,
                   force_exit ? c->d_force_exit : nullptr, false, debug);
}

// Copy a matrix given in canonical layout into a row range of a repacked one.
int copy_rows(ee_ctx* c, void* dst, size_t dst_pitch, const void* src, size_t src_pitch,
              size_t row_bytes, size_t rows) {
  HIPCHK(c, hipMemcpy2D(dst, dst_pitch, src, src_pitch, row_bytes, rows, hipMemcpyDefault));
  return EE_OK;
}

// q or k heads: pair-interleave rows (i, i + D/2) of every head.
int copy_rope_heads(ee_ctx* c, char* dst, const char* src, int heads) {
  const int D = c->cfg.head_dim;
  const size_t rb = static_cast<size_t>(c->cfg.hidden) * c->esz;
  int r;
  for (int h = 0; h < heads; ++h) {
    char* d = dst + static_cast<size_t>(h) * D * rb;
    const char* s = src + static_cast<size_t>(h) * D * rb;
    if ((r = copy_rows(c, d, 2 * rb, s, rb, rb, D / 2))) return r;
    if ((r = copy_rows(c, d + rb, 2 * rb, s + (D / 2) * rb, rb, rb, D / 2))) return r;
  }
  return EE_OK;
}

int load_one(ee_ctx* c, const ee_tensor& t) {
  const ee_config& g = c->cfg;
  const int64_t H = g.hidden, A = g.n_q_heads, K = g.n_kv_heads, D = g.head_dim, F = g.ffn,
                V = g.vocab;
  const int64_t es = static_cast<int64_t>(c->esz);
  if (!t.name || !t.ptr) return fail(c, EE_EINVAL, "tensor with null name or pointer");
  const std::string name(t.name);
  auto need = [&](int64_t bytes) -> int {
    if (t.nbytes != bytes)
      return fail(c, EE_EINVAL, "tensor " + name + ": nbytes " + std::to_string(t.nbytes) +
                                    ", expected " + std::to_string(bytes));
    return EE_OK;
  };
  int r;
  if (name == "embed") {
    if ((r = need(V * H * es))) return r;
    HIPCHK(c, hipMemcpy(c->embed, t.ptr, t.nbytes, hipMemcpyDefault));
  } else if (name == "final_norm") {
    if ((r = need(H * 4))) return r;
    HIPCHK(c, hipMemcpy(c->g_final, t.ptr, t.nbytes, hipMemcpyDefault));
  } else if (name.rfind("layers.", 0) == 0) {
    const size_t dot = name.find('.', 7);
    if (dot == std::string::npos) return fail(c, EE_EINVAL, "bad tensor name " + name);
    const int l = atoi(name.substr(7, dot - 7).c_str());
    const std::string leaf = name.substr(dot + 1);
    if (l < 0 || l >= g.n_layers || name.substr(7, dot - 7) != std::to_string(l))
      return fail(c, EE_EINVAL, "bad layer index in " + name);
    const size_t rb = static_cast<size_t>(H * es);
    char* qkv = static_cast<char*>(c->wqkv[l]);
    const char* src = static_cast<const char*>(t.ptr);
    if (leaf == "attn_norm" || leaf == "mlp_norm") {
      if ((r = need(H * 4))) return r;
      HIPCHK(c, hipMemcpy(leaf == "attn_norm" ? c->g_attn[l] : c->g_mlp[l], t.ptr, t.nbytes,
                          hipMemcpyDefault));
    } else if (leaf == "wq") {
      if ((r = need(A * D * H * es))) return r;
      if ((r = copy_rope_heads(c, qkv, src, static_cast<int>(A)))) return r;
    } else if (leaf == "wk") {
      if ((r = need(K * D * H * es))) return r;
      if ((r = copy_rope_heads(c, qkv + A * D * rb, src, static_cast<int>(K)))) return r;
    } else if (leaf == "wv") {
      if ((r = need(K * D * H * es))) return r;
      HIPCHK(c, hipMemcpy(qkv + (A + K) * D * rb, t.ptr, t.nbytes, hipMemcpyDefault));
    } else if (leaf == "wo") {
      if ((r = need(H * A * D * es))) return r;
      HIPCHK(c, hipMemcpy(c->wo[l], t.ptr, t.nbytes, hipMemcpyDefault));
    } else if (leaf == "w_gate" || leaf == "w_up") {
      if ((r = need(F * H * es))) return r;
      char* dst = static_cast<char*>(c->wgu[l]) + (leaf == "w_up" ? rb : 0);
      if ((r = copy_rows(c, dst, 2 * rb, src, rb, rb, static_cast<size_t>(F)))) return r;
    } else if (leaf == "w_down") {
      if ((r = need(H * F * es))) return r;
      HIPCHK(c, hipMemcpy(c->wd[l], t.ptr, t.nbytes, hipMemcpyDefault));
    } else {
      return fail(c, EE_EINVAL, "unknown tensor " + name);
    }
  } else if (name.rfind("readout.", 0) == 0) {
    const size_t dot = name.find('.', 8);
    if (dot == std::string::npos) return fail(c, EE_EINVAL, "bad tensor name " + name);
    const int L = atoi(name.substr(8, dot - 8).c_str());
    const std::string leaf = name.substr(dot + 1);
    if (L < 1 || L > g.n_layers || name.substr(8, dot - 8) != std::to_string(L))
      return fail(c, EE_EINVAL, "readout layer must be 1..n_layers in " + name);
    if (leaf != "w" && leaf != "b") return fail(c, EE_EINVAL, "unknown tensor " + name);
    if ((r = need(leaf == "w" ? H * H * es : H * 4))) return r;
    if (!c->readout.count(L)) {
      void* w = nullptr;
      float* b = nullptr;
      if ((r = dalloc(c, &w, static_cast<size_t>(H * H * es)))) return r;
      if ((r = dalloc(c, &b, static_cast<size_t>(H * 4)))) {
        dfree(w);
        return r;
      }
      c->readout[L] = {w, b};
    }
    auto& ro = c->readout[L];
    HIPCHK(c, hipMemcpy(leaf == "w" ? ro.first : static_cast<void*>(ro.second), t.ptr, t.nbytes,
                        hipMemcpyDefault));
    return EE_OK;  // readouts are not part of the required set
  } else {
    return fail(c, EE_EINVAL, "unknown tensor " + name);
  }
  c->loaded.insert(name);
  return EE_OK;
}

}  // namespace

extern "C" {

static int create_body(ee_ctx* c, const ee_config* cfg, void* hip_stream, ee_ctx** out);

static int create_impl(const ee_config* cfg, void* hip_stream, ee_ctx** out) {
  if (!cfg || !out) return EE_EINVAL;
  *out = nullptr;
  std::string why;
  g_create_err.clear();
  if (!validate_config(cfg, why)) {
    g_create_err = why;
    return EE_EINVAL;
  }
  ee_ctx* c = new (std::nothrow) ee_ctx();
  if (!c) {
    g_create_err = "out of host memory";
    return EE_ENOMEM;
  }
  try {
    return create_body(c, cfg, hip_stream, out);
  } catch (...) {
    ee_destroy(c);
    throw;
  }
}

static int create_body(ee_ctx* c, const ee_config* cfg, void* hip_stream, ee_ctx** out) {
  c->cfg = *cfg;
  c->wbf16 = cfg->wdtype == EE_BF16;
  c->esz = c->wbf16 ? 2 : 4;
  int r = EE_OK;
  auto bail = [&](int code) {
    g_create_err = c->err.empty() ? "ee_create failed" : c->err;
    ee_destroy(c);
    return code;
  };
  hipError_t he;
  if ((he = hipGetDevice(&c->device)) != hipSuccess) return bail(hip_fail(c, he, "hipGetDevice"));
  if ((he = hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device)) != hipSuccess)
    return bail(hip_fail(c, he, "hipDeviceGetAttribute"));
  if ((he = ee::scratch_address(c->device, &c->scratch)) != hipSuccess)
    return bail(hip_fail(c, he, "hipGetSymbolAddress of the library scratch"));
  if (hip_stream) {
    c->stream = static_cast<hipStream_t>(hip_stream);
  } else {
    if ((he = hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking)) != hipSuccess)
      return bail(hip_fail(c, he, "hipStreamCreateWithFlags"));
    c->own_stream = true;
  }
  if ((he = hipEventCreate(&c->ev0)) != hipSuccess || (he = hipEventCreate(&c->ev1)) != hipSuccess)
    return bail(hip_fail(c, he, "hipEventCreate"));
  const ee_config& g = *cfg;
  const size_t es = c->esz;
  const size_t H = g.hidden, A = g.n_q_heads, K = g.n_kv_heads, D = g.head_dim, F = g.ffn,
               V = g.vocab, L = g.n_layers;
  if ((r = dalloc(c, &c->embed, V * H * es))) return bail(r);
  c->wqkv.assign(L, nullptr); c->wo.assign(L, nullptr); c->wgu.assign(L, nullptr);
  c->wd.assign(L, nullptr); c->g_attn.assign(L, nullptr); c->g_mlp.assign(L, nullptr);
  for (size_t l = 0; l < L; ++l) {
    if ((r = dalloc(c, &c->wqkv[l], (A + 2 * K) * D * H * es))) return bail(r);
    if ((r = dalloc(c, &c->wo[l], H * A * D * es))) return bail(r);
    if ((r = dalloc(c, &c->wgu[l], 2 * F * H * es))) return bail(r);
    if ((r = dalloc(c, &c->wd[l], H * F * es))) return bail(r);
    if ((r = dalloc(c, &c->g_attn[l], H * 4))) return bail(r);
    if ((r = dalloc(c, &c->g_mlp[l], H * 4))) return bail(r);
  }
  if ((r = dalloc(c, &c->g_final, H * 4))) return bail(r);
  if ((r = dalloc(c, &c->d_layers, L * sizeof(ee::LayerW)))) return bail(r);
  {
    std::vector<ee::LayerW> lw(L);
    for (size_t l = 0; l < L; ++l)
      lw[l] = ee::LayerW{c->wqkv[l], c->wo[l], c->wgu[l], c->wd[l], c->g_attn[l], c->g_mlp[l]};
    if ((he = hipMemcpy(c->d_layers, lw.data(), L * sizeof(ee::LayerW), hipMemcpyHostToDevice)) != hipSuccess)
      return bail(hip_fail(c, he, "hipMemcpy layer table"));
    c->h_layers = lw;
  }
  c->n_pages = (g.max_seq + g.page_size - 1) / g.page_size;
  c->layer_stride = static_cast<int64_t>(c->n_pages) * K * g.page_size * D;
  if ((r = dalloc(c, &c->kpool, L * c->layer_stride * es))) return bail(r);
  if ((r = dalloc(c, &c->vpool, L * c->layer_stride * es))) return bail(r);
  if ((r = dalloc(c, &c->d_block_table, sizeof(int32_t) * c->n_pages))) return bail(r);
  if ((he = hipHostMalloc(reinterpret_cast<void**>(&c->h_block_table), sizeof(int32_t) * c->n_pages)) != hipSuccess)
    return bail(hip_fail(c, he, "hipHostMalloc block table"));
  reset_pages(c);
  // RoPE: angle = pos * base^(-2i/D), computed in double, stored as float.
  {
    const size_t half = D / 2;
    std::vector<float> cs(static_cast<size_t>(g.max_seq) * half), sn(cs.size());
    for (int t = 0; t < g.max_seq; ++t)
      for (size_t i = 0; i < half; ++i) {
        const double inv = pow(static_cast<double>(g.rope_base), -2.0 * static_cast<double>(i) / D);
        const double ang = static_cast<double>(t) * inv;
        cs[t * half + i] = static_cast<float>(cos(ang));
        sn[t * half + i] = static_cast<float>(sin(ang));
      }
    if ((r = dalloc(c, &c->d_cos, cs.size() * 4))) return bail(r);
    if ((r = dalloc(c, &c->d_sin, sn.size() * 4))) return bail(r);
    if ((he = hipMemcpy(c->d_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice)) != hipSuccess ||
        (he = hipMemcpy(c->d_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice)) != hipSuccess)
      return bail(hip_fail(c, he, "hipMemcpy rope tables"));
  }
  c->max_splits = (g.max_seq + ee::kAttnSplit - 1) / ee::kAttnSplit;
  {
    int64_t off[kTwParts];
    const int64_t total = tw_layout(g, off);
    uint64_t** const ptrs[kTwParts] = {&c->d_h, &c->d_hexit, &c->d_z, &c->d_q, &c->d_o, &c->d_a,
                                       &c->d_kvnew, &c->d_dec, &c->d_attn_part};
    if ((r = dalloc(c, &c->d_tw, total * 8)) || (r = dalloc(c, &c->d_x, H * 4))) return bail(r);
    c->tw_words = total;
    tw_bind(c->d_tw, off, ptrs);
    if ((he = hipMemset(c->d_tw, 0, total * 8)) != hipSuccess) return bail(hip_fail(c, he, "hipMemset"));
  }
  if ((r = dalloc(c, &c->d_hist, sizeof(int32_t) * g.max_seq))) return bail(r);
  {
    // chunks of up to 1024 positions: the residual stream, queries, attention
    // output and feed-forward activations of a chunk, and the split workspaces
    ee::BatchBuffers& b = c->bbuf;
    const size_t Pm = static_cast<size_t>(std::min(1024, g.max_seq));
    const size_t nmax = std::max({(A + 2 * K) * D, 2 * F, H});
    b.max_positions = static_cast<int>(Pm);
    b.gemm_ws_floats = std::min<size_t>(size_t(8) << 20, 32 * Pm * nmax);
    b.attn_ws_floats = std::min<size_t>(size_t(8) << 20, 16 * Pm * A * (D + 2));
    b.n_tile_ctr = ee::batch_tile_counters(static_cast<int>(Pm), static_cast<int>(nmax));
    if ((r = dalloc(c, &b.X, Pm * H * 4)) || (r = dalloc(c, &b.Q, Pm * A * D * 4)) ||
        (r = dalloc(c, &b.O, Pm * A * D * 4)) || (r = dalloc(c, &b.Act, Pm * F * 4)) ||
        (r = dalloc(c, &b.gemm_ws, b.gemm_ws_floats * 4)) || (r = dalloc(c, &b.attn_ws, b.attn_ws_floats * 4)) ||
        (r = dalloc(c, &b.tile_ctr, b.n_tile_ctr * 4)))
      return bail(r);
  }
  if ((r = dalloc(c, &c->d_counters, sizeof(ee::Counters)))) return bail(r);
  if ((r = dalloc(c, &c->d_ctl, sizeof(ee::StepCtl)))) return bail(r);

  DevParams p = make_params(c, INFINITY, 0);
  c->lds = ee::lds_bytes(p);
  c->fill_slots = ee::fill_batch_slots(p);
  const int cpl = ee::chunks_per_lane(p, c->wbf16);
  if (cpl > (c->wbf16 ? 4 : 2)) {
    c->err = "hidden too large for the compiled kernels (bf16: H <= 2048, fp32: H <= 512)";
    return bail(EE_EINVAL);
  }
  if (c->lds > 64 * 1024) {
    c->err = "shape needs more than 64 KB of LDS per workgroup";
    return bail(EE_EINVAL);
  }
  c->max_wgs_per_cu = ee::persistent_max_wgs_per_cu(p, c->wbf16, c->lds);
  c->slot = take_slot();
  if ((he = hipHostMalloc(reinterpret_cast<void**>(&c->params_pinned), sizeof(DevParams))) != hipSuccess)
    return bail(hip_fail(c, he, "hipHostMalloc parameter block"));
  // without a free parameter slot the context uses the one-kernel-per-operation program
  c->nwg_persistent = (c->max_wgs_per_cu > 0 && c->slot >= 0) ? c->n_cu * c->max_wgs_per_cu : 0;
  c->persistent = c->nwg_persistent > 0;
  c->head_wgs = 2 * c->n_cu;
  c->max_parts = std::max(c->head_wgs, c->nwg_persistent);
  if ((r = dalloc(c, &c->d_head_part, static_cast<size_t>(c->max_parts) * ee::kStatFloats * 4))) return bail(r);
  *out = c;
  return EE_OK;
}

static int load_weights_impl(ee_ctx* c, const ee_tensor* tensors, int32_t n_tensors) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (!tensors || n_tensors < 0) return fail(c, EE_EINVAL, "bad tensor list");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  for (int i = 0; i < n_tensors; ++i) {
    const int r = load_one(c, tensors[i]);
    if (r) return r;
  }
  HIPCHK(c, hipDeviceSynchronize());
  return EE_OK;
}

// Full depth over positions pos .. pos + n - 1 with device input tokens
// d_tokens, batched (chunks of positions through each layer together); with
// head, the final head of the last position sets the next input token.
// Advances the position; synchronous.
static int batched_full_depth(ee_ctx* c, const int32_t* d_tokens, int n, bool head) {
  int r;
  if ((r = ensure_pages(c, c->pos + n))) return r;
  ee::BatchPass bp{};
  bp.p = make_params(c, INFINITY, 0);
  bp.layers = c->h_layers.data();
  bp.buf = c->bbuf;
  if (c->prefill_chunk > 0) bp.buf.max_positions = std::min(c->prefill_chunk, c->bbuf.max_positions);
  bp.wbf16 = c->wbf16;
  bp.n_cu = c->n_cu;
  HIPCHK(c, hipMemsetAsync(reinterpret_cast<char*>(c->d_ctl) + offsetof(ee::StepCtl, exited), 0,
                           offsetof(ee::StepCtl, pad) - offsetof(ee::StepCtl, exited), c->stream));
  HIPCHK(c, hipEventRecord(c->ev0, c->stream));
  hipError_t e = ee::launch_batched_pass(bp, c->pos, d_tokens, n, c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "batched pass launch");
  if (head) {
    const int Pm = bp.buf.max_positions;
    const int last = (n - 1) % Pm;  // row of the last position in the last chunk
    e = ee::launch_head_eval(make_params(c, INFINITY, 0), c->wbf16,
                             bp.buf.X + static_cast<size_t>(last) * c->cfg.hidden, 0, c->head_wgs, c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "prompt head launch");
  }
  HIPCHK(c, hipEventRecord(c->ev1, c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  HIPCHK(c, hipEventElapsedTime(&c->last_ms, c->ev0, c->ev1));
  ee::StepCtl ctl;
  HIPCHK(c, hipMemcpy(&ctl, c->d_ctl, sizeof(ctl), hipMemcpyDeviceToHost));
  if (ctl.error != ee::kErrNone) {
    c->have_next = false;
    return fail(c, EE_EDEVICE, "device: token id out of range");
  }
  c->pos += n;
  return EE_OK;
}

static int prefill_impl(ee_ctx* c, const int32_t* tokens, int32_t n, int32_t* out_first_token) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (!weights_ready(c)) return fail(c, EE_ESTATE, "weights not fully loaded");
  if (!tokens || n <= 0) return fail(c, EE_EINVAL, "prefill needs at least one token");
  int r;
  if ((r = upload_force(c, n, tokens, nullptr))) return r;
  if (c->prefill_chunk != 0) {
    if ((r = batched_full_depth(c, c->d_force_tok, n, true))) return r;
    c->have_next = true;
  } else if ((r = run_steps(c, INFINITY, 0, n, c->d_force_tok, nullptr, true, false))) {
    return r;
  }
  int32_t tok = -1;
  HIPCHK(c, hipMemcpy(&tok, &c->d_ctl->next_token, sizeof(tok), hipMemcpyDeviceToHost));
  if (out_first_token) *out_first_token = tok;
  return EE_OK;
}

static int refresh_impl(ee_ctx* c, int32_t n) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (!weights_ready(c)) return fail(c, EE_ESTATE, "weights not fully loaded");
  if (n < 1 || n > c->pos) return fail(c, EE_EINVAL, "refresh needs 1 <= n <= position");
  int r;
  if ((r = ensure_force(c, n))) return r;
  HIPCHK(c, hipMemcpyAsync(c->d_force_tok, c->d_hist + (c->pos - n), sizeof(int32_t) * n,
                           hipMemcpyDeviceToDevice, c->stream));
  int32_t next = 0;
  HIPCHK(c, hipMemcpy(&next, &c->d_ctl->next_token, sizeof(next), hipMemcpyDeviceToHost));
  const bool had = c->have_next;
  c->pos -= n;
  r = c->prefill_chunk != 0 ? batched_full_depth(c, c->d_force_tok, n, false)
                            : run_steps(c, INFINITY, 0, n, c->d_force_tok, nullptr, true, false);
  if (r) {
    c->pos += n;
    c->have_next = false;
    return r;
  }
  // the pass's own head output is not an emitted token: the next input stays
  HIPCHK(c, hipMemcpy(&c->d_ctl->next_token, &next, sizeof(next), hipMemcpyHostToDevice));
  c->have_next = had;
  return EE_OK;
}

static int decode_n_ex_impl(ee_ctx* c, float tau, int32_t exit_layer, int32_t n, const int32_t* force_tokens,
                   const int32_t* force_exit, int32_t* tokens, int32_t* exited, float* conf,
                   int32_t* would_exit) {
  int r = decode_common(c, tau, exit_layer, n, force_tokens, force_exit, false);
  if (r) return r;
  return copy_ring(c, n, tokens, exited, conf, would_exit);
}

static int decode_n_impl(ee_ctx* c, float tau, int32_t exit_layer, int32_t n, int32_t* tokens,
                int32_t* exited, float* conf) {
  return ee_decode_n_ex(c, tau, exit_layer, n, nullptr, nullptr, tokens, exited, conf, nullptr);
}

static int decode_n_noalloc_impl(ee_ctx* c, float tau, int32_t exit_layer, int32_t n, int32_t* d_tokens,
                                 int32_t* d_exited, float* d_conf) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (n <= 0) return fail(c, EE_EINVAL, "n must be positive");
  if (!d_tokens || !d_exited || !d_conf) return fail(c, EE_EINVAL, "output arrays must be non-null device pointers");
  int r;
  if ((r = check_gate_args(c, tau, exit_layer))) return r;
  if (!c->have_next) return fail(c, EE_ESTATE, "no input token: run ee_prefill first");
  if (!c->scratch) return fail(c, EE_ESTATE, "no library scratch on this device");
  const NoAlloc na{d_tokens, d_exited, d_conf};
  return run_steps(c, tau, exit_layer, n, nullptr, nullptr, false, false, &na);
}

static int decode_step_impl(ee_ctx* c, float tau, int32_t exit_layer, int32_t* out_token,
                   int32_t* out_exited, float* out_conf) {
  return ee_decode_n_ex(c, tau, exit_layer, 1, nullptr, nullptr, out_token, out_exited, out_conf,
                        nullptr);
}

static int decode_step_ex_impl(ee_ctx* c, float tau, int32_t exit_layer, int32_t input_token,
                      int32_t force_exit, ee_debug* dbg) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  int r;
  const bool want_logits = dbg && (dbg->logits_readout || dbg->logits_full);
  if (want_logits && !c->d_dbg_r) {
    if ((r = dalloc(c, &c->d_dbg_r, static_cast<size_t>(c->cfg.vocab) * 4))) return r;
    if ((r = dalloc(c, &c->d_dbg_f, static_cast<size_t>(c->cfg.vocab) * 4))) return r;
  }
  const int32_t ft[1] = {input_token};
  const int32_t fe[1] = {force_exit};
  c->nucleus = dbg != nullptr;
  r = decode_common(c, tau, exit_layer, 1, input_token >= 0 ? ft : nullptr,
                    force_exit >= 0 ? fe : nullptr, want_logits);
  c->nucleus = false;
  if (r) return r;
  if (!dbg) return EE_OK;
  ee::StepCtl ctl;
  HIPCHK(c, hipMemcpy(&ctl, c->d_ctl, sizeof(ctl), hipMemcpyDeviceToHost));
  int32_t tok = 0, ex = 0, would = 0;
  float cf = 0.f;
  if ((r = copy_ring(c, 1, &tok, &ex, &cf, &would))) return r;
  const size_t H = c->cfg.hidden, V = c->cfg.vocab;
  dbg->token = tok;
  dbg->exited = ex;
  dbg->would_exit = would;
  dbg->conf = cf;
  dbg->readout_token = exit_layer > 0 ? ctl.readout_token : -1;
  dbg->full_token = ex ? -1 : ctl.full_token;
  dbg->conf_full = ex ? NAN : ctl.conf_full;
  dbg->nucleus_mass = NAN;
  if (!ex && exit_layer > 0)
    HIPCHK(c, hipMemcpy(&dbg->nucleus_mass, c->d_ring_mass, sizeof(float), hipMemcpyDeviceToHost));
  if (dbg->h_exit && exit_layer > 0 && (r = copy_untag(c, dbg->h_exit, c->d_hexit, H))) return r;
  if (dbg->h_final && !ex && (r = copy_untag(c, dbg->h_final, c->d_h, H))) return r;
  if (dbg->logits_readout && exit_layer > 0)
    HIPCHK(c, hipMemcpy(dbg->logits_readout, c->d_dbg_r, V * 4, hipMemcpyDeviceToHost));
  if (dbg->logits_full && !ex)
    HIPCHK(c, hipMemcpy(dbg->logits_full, c->d_dbg_f, V * 4, hipMemcpyDeviceToHost));
  return EE_OK;
}

static int calibrate_threshold_impl(ee_ctx* c, const int32_t* prompts, const int32_t* prompt_lens,
                           int32_t n_prompts, int32_t n_gen, int32_t exit_layer, int32_t mode,
                           float target, float* out_tau) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (!prompts || !prompt_lens || n_prompts <= 0 || n_gen <= 0 || !out_tau)
    return fail(c, EE_EINVAL, "calibration needs prompts, n_gen > 0 and an output");
  if (exit_layer < 1) return fail(c, EE_EINVAL, "calibration needs a gated exit layer");
  if (mode != EE_CAL_EXIT_RATE && mode != EE_CAL_MEDIAN && mode != EE_CAL_NUCLEUS)
    return fail(c, EE_EINVAL, "unknown mode");
  if (mode != EE_CAL_MEDIAN && !(target >= 0.f && target <= 1.f))
    return fail(c, EE_EINVAL, "target must be in [0, 1]");
  int r;
  if ((r = check_gate_args(c, INFINITY, exit_layer))) return r;
  std::vector<float> confs, masses;
  std::vector<float> buf(n_gen), mbuf(n_gen);
  size_t off = 0;
  for (int i = 0; i < n_prompts; ++i) {
    if (prompt_lens[i] <= 0) return fail(c, EE_EINVAL, "empty calibration prompt");
    if ((r = ee_reset(c))) return r;
    int32_t first = 0;
    if ((r = ee_prefill(c, prompts + off, prompt_lens[i], &first))) return r;
    c->nucleus = mode == EE_CAL_NUCLEUS;
    r = ee_decode_n(c, INFINITY, exit_layer, n_gen, nullptr, nullptr, buf.data());
    c->nucleus = false;
    if (r) return r;
    confs.insert(confs.end(), buf.begin(), buf.end());
    if (mode == EE_CAL_NUCLEUS) {
      HIPCHK(c, hipMemcpy(mbuf.data(), c->d_ring_mass, sizeof(float) * n_gen, hipMemcpyDeviceToHost));
      masses.insert(masses.end(), mbuf.begin(), mbuf.end());
    }
    off += prompt_lens[i];
  }
  if ((r = ee_reset(c))) return r;
  c->cal_confs = confs;
  c->cal_masses = masses;
  if (mode != EE_CAL_NUCLEUS) c->cal_masses.assign(confs.size(), NAN);
  if (mode == EE_CAL_NUCLEUS) {
    // the lowest grid threshold whose early answers are acceptable often enough
    *out_tau = INFINITY;
    for (int g = 0; g < 100; ++g) {
      const float tau = static_cast<float>(g / 100.0);
      size_t early = 0, ok = 0;
      for (size_t i = 0; i < confs.size(); ++i) {
        if (confs[i] > tau) {
          ++early;
          ok += masses[i] < kNucleusTopP;
        }
      }
      if (early > 0 && static_cast<double>(ok) / static_cast<double>(early) >= static_cast<double>(target)) {
        *out_tau = tau;
        break;
      }
    }
    return EE_OK;
  }
  std::sort(confs.begin(), confs.end());
  const size_t n = confs.size();
  if (mode == EE_CAL_MEDIAN) {
    const double med = n % 2 ? confs[n / 2]
                             : 0.5 * (static_cast<double>(confs[n / 2 - 1]) + confs[n / 2]);
    *out_tau = static_cast<float>(med);
  } else {
    const size_t k = static_cast<size_t>(floor(static_cast<double>(target) * n + 0.5));
    if (k == 0) *out_tau = INFINITY;
    else if (k >= n) *out_tau = -INFINITY;
    else *out_tau = confs[n - k - 1];
  }
  return EE_OK;
}

static int calibration_record_impl(ee_ctx* c, int32_t n, float* confs, float* masses) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (c->cal_confs.empty()) return fail(c, EE_ESTATE, "no calibration has run on this context");
  if (n != static_cast<int32_t>(c->cal_confs.size()))
    return fail(c, EE_EINVAL, "the latest calibration recorded " + std::to_string(c->cal_confs.size()) + " steps");
  if (confs) memcpy(confs, c->cal_confs.data(), sizeof(float) * n);
  if (masses) memcpy(masses, c->cal_masses.data(), sizeof(float) * n);
  return EE_OK;
}

static int set_readout_bias_impl(ee_ctx* c, int32_t exit_layer, const float* b, int32_t on_device) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  auto it = c->readout.find(exit_layer);
  if (it == c->readout.end() || !b) return fail(c, EE_EINVAL, "no readout at that layer");
  HIPCHK(c, hipMemcpyAsync(it->second.second, b, sizeof(float) * c->cfg.hidden,
                           on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice, c->stream));
  return EE_OK;
}

static int set_prefill_chunk_impl(ee_ctx* c, int32_t positions) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (positions < 0) return fail(c, EE_EINVAL, "positions must be >= 0");
  c->prefill_chunk = positions == 0 ? 0 : std::min(positions, c->bbuf.max_positions);
  return EE_OK;
}

static int set_fill_policy_impl(ee_ctx* c, int32_t policy) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (policy != EE_FILL_EAGER && policy != EE_FILL_LAZY) return fail(c, EE_EINVAL, "unknown fill policy");
  c->fill_lazy = policy == EE_FILL_LAZY;
  return EE_OK;
}

static int stream_probe_impl(ee_ctx* c, int64_t bytes, int32_t reps, float* out_gbps) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (!out_gbps || bytes < 16 || reps < 1) return fail(c, EE_EINVAL, "stream probe: bytes >= 16, reps >= 1, output");
  const int64_t n = bytes / 16;
  void* buf = nullptr;
  uint32_t* sink = nullptr;
  int r;
  if ((r = dalloc(c, &buf, static_cast<size_t>(n) * 16))) return r;
  if ((r = dalloc(c, reinterpret_cast<void**>(&sink), 4))) {
    dfree(buf);
    return r;
  }
  std::vector<float> ms;
  hipError_t he = hipMemsetAsync(buf, 0, static_cast<size_t>(n) * 16, c->stream);
  for (int i = 0; i <= reps && he == hipSuccess; ++i) {  // launch 0 warms up
    if ((he = hipEventRecord(c->ev0, c->stream)) != hipSuccess) break;
    if ((he = ee::launch_stream_read(buf, n, c->n_cu, sink, c->stream)) != hipSuccess) break;
    if ((he = hipEventRecord(c->ev1, c->stream)) != hipSuccess) break;
    if ((he = hipEventSynchronize(c->ev1)) != hipSuccess) break;
    float t = 0.f;
    if ((he = hipEventElapsedTime(&t, c->ev0, c->ev1)) != hipSuccess) break;
    if (i > 0) ms.push_back(t);
  }
  dfree(buf);
  dfree(sink);
  if (he != hipSuccess) return hip_fail(c, he, "stream probe");
  std::sort(ms.begin(), ms.end());
  const float med = ms[ms.size() / 2];
  *out_gbps = static_cast<float>(static_cast<double>(n) * 16.0 / (med * 1e-3) / 1e9);
  return EE_OK;
}

static int set_confidence_measure_impl(ee_ctx* c, int32_t measure) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (measure != EE_CONF_MAXPROB && measure != EE_CONF_MARGIN && measure != EE_CONF_NEGENTROPY)
    return fail(c, EE_EINVAL, "unknown confidence measure");
  c->conf_measure = measure;
  return EE_OK;
}

static int head_eval_impl(ee_ctx* c, int32_t readout_layer, const float* x, int32_t* out_token,
                 float* out_conf, float* out_logits) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (!x) return fail(c, EE_EINVAL, "x is null");
  int r;
  if ((r = check_gate_args(c, INFINITY, readout_layer))) return r;
  if (out_logits && !c->d_dbg_r) {
    if ((r = dalloc(c, &c->d_dbg_r, static_cast<size_t>(c->cfg.vocab) * 4))) return r;
    if ((r = dalloc(c, &c->d_dbg_f, static_cast<size_t>(c->cfg.vocab) * 4))) return r;
  }
  HIPCHK(c, hipMemcpyAsync(c->d_x, x, sizeof(float) * c->cfg.hidden, hipMemcpyHostToDevice, c->stream));
  DevParams p = make_params(c, INFINITY, readout_layer);
  if (out_logits) {
    p.dbg_logits_r = c->d_dbg_r;
    p.dbg_logits_f = c->d_dbg_f;
  }
  ee::StepCtl saved;
  HIPCHK(c, hipMemcpy(&saved, c->d_ctl, sizeof(saved), hipMemcpyDeviceToHost));
  HIPCHK(c, hipMemsetAsync(reinterpret_cast<char*>(c->d_ctl) + offsetof(ee::StepCtl, exited), 0,
                           offsetof(ee::StepCtl, pad) - offsetof(ee::StepCtl, exited), c->stream));
  hipError_t e = ee::launch_head_eval(p, c->wbf16, c->d_x, readout_layer > 0, c->head_wgs, c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "head eval launch");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  ee::StepCtl ctl;
  HIPCHK(c, hipMemcpy(&ctl, c->d_ctl, sizeof(ctl), hipMemcpyDeviceToHost));
  // the eval's head wrote next_token: restore the sequence's
  HIPCHK(c, hipMemcpy(&c->d_ctl->next_token, &saved.next_token, sizeof(int32_t), hipMemcpyHostToDevice));
  if (out_token) *out_token = readout_layer > 0 ? ctl.readout_token : ctl.full_token;
  if (out_conf) *out_conf = readout_layer > 0 ? ctl.conf : ctl.conf_full;
  if (out_logits)
    HIPCHK(c, hipMemcpy(out_logits, readout_layer > 0 ? c->d_dbg_r : c->d_dbg_f,
                        sizeof(float) * c->cfg.vocab, hipMemcpyDeviceToHost));
  return EE_OK;
}

static int read_kv_impl(ee_ctx* c, int32_t layer, int32_t pos, float* k_out, float* v_out) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (layer < 0 || layer >= c->cfg.n_layers || pos < 0 || pos >= c->pos)
    return fail(c, EE_EINVAL, "layer or position out of range");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  const int K = c->cfg.n_kv_heads, D = c->cfg.head_dim, P = c->cfg.page_size;
  const int page = c->h_block_table[pos / P], slot = pos % P;
  std::vector<unsigned char> buf(static_cast<size_t>(D) * c->esz);
  for (int pass = 0; pass < 2; ++pass) {
    float* out = pass ? v_out : k_out;
    if (!out) continue;
    const char* pool = static_cast<const char*>(pass ? c->vpool : c->kpool);
    for (int h = 0; h < K; ++h) {
      const int64_t off = static_cast<int64_t>(layer) * c->layer_stride +
                          ((static_cast<int64_t>(page) * K + h) * P + slot) * D;
      HIPCHK(c, hipMemcpy(buf.data(), pool + off * c->esz, buf.size(), hipMemcpyDeviceToHost));
      for (int d = 0; d < D; ++d) {
        float f;
        if (c->wbf16) {
          uint16_t b;
          memcpy(&b, buf.data() + 2 * d, 2);
          const uint32_t u = static_cast<uint32_t>(b) << 16;
          memcpy(&f, &u, 4);
        } else {
          memcpy(&f, buf.data() + 4 * d, 4);
        }
        // keys are stored with rotate-half pairs interleaved: element 2i is
        // dimension i, element 2i+1 is dimension i + D/2
        const int dim = pass ? d : ((d & 1) ? D / 2 + d / 2 : d / 2);
        out[h * D + dim] = f;
      }
    }
  }
  return EE_OK;
}

static int set_persistent_impl(ee_ctx* c, int32_t wgs_per_cu) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (wgs_per_cu == 0) {
    c->persistent = false;
    return EE_OK;
  }
  if (wgs_per_cu < 0) wgs_per_cu = std::max(1, c->max_wgs_per_cu);
  if (wgs_per_cu > c->max_wgs_per_cu)
    return fail(c, EE_EINVAL, "at most " + std::to_string(c->max_wgs_per_cu) +
                                  " persistent workgroups per CU can be co-resident");
  if (c->slot < 0) return fail(c, EE_ESTATE, "no free persistent-kernel parameter slot");
  c->persistent = true;
  c->nwg_persistent = c->n_cu * wgs_per_cu;
  return EE_OK;
}

static int set_persistent_grid_impl(ee_ctx* c, int32_t nwg) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  const int most = std::min(c->max_parts, c->n_cu * c->max_wgs_per_cu);
  if (nwg < 1 || nwg > most)
    return fail(c, EE_EINVAL, "persistent grid must hold 1.." + std::to_string(most) + " workgroups");
  if (c->slot < 0) return fail(c, EE_ESTATE, "no free persistent-kernel parameter slot");
  c->persistent = true;
  c->nwg_persistent = nwg;
  return EE_OK;
}

static int set_timeline_impl(ee_ctx* c, int32_t capacity) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  if (capacity < 0) return fail(c, EE_EINVAL, "capacity must be >= 0");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  dfree(c->d_timeline);
  c->d_timeline = nullptr;
  c->timeline_cap = 0;
  if (capacity > 0) {
    int r;
    if ((r = dalloc(c, &c->d_timeline, sizeof(uint64_t) * capacity))) return r;
    c->timeline_cap = capacity;
  }
  return EE_OK;
}

static int read_timeline_impl(ee_ctx* c, uint64_t* out, int32_t n) {
  if (!c || !out || n < 0) return EE_EINVAL;
  c->err.clear();
  if (n > c->timeline_cap) return fail(c, EE_EINVAL, "more entries requested than recorded");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  HIPCHK(c, hipMemcpy(out, c->d_timeline, sizeof(uint64_t) * n, hipMemcpyDeviceToHost));
  return EE_OK;
}

static int last_decode_ms_impl(ee_ctx* c, float* out_ms) {
  if (!c || !out_ms) return EE_EINVAL;
  *out_ms = c->last_ms;
  return EE_OK;
}

int32_t ee_position(const ee_ctx* c) { return c ? c->pos : -1; }

static int reset_impl(ee_ctx* c) {
  if (!c) return EE_EINVAL;
  c->err.clear();
  HIPCHK(c, hipStreamSynchronize(c->stream));
  c->pos = 0;
  c->have_next = false;
  reset_pages(c);
  HIPCHK(c, hipMemset(c->d_ctl, 0, sizeof(ee::StepCtl)));
  HIPCHK(c, hipMemset(c->d_counters, 0, sizeof(ee::Counters)));
  HIPCHK(c, hipDeviceSynchronize());
  return EE_OK;
}

const char* ee_last_error(const ee_ctx* c) { return c ? c->err.c_str() : g_create_err.c_str(); }

static void destroy_impl(ee_ctx* c) {
  if (!c) return;
  if (c->stream) (void)hipStreamSynchronize(c->stream);
  dfree(c->embed);
  for (void* p : c->wqkv) dfree(p);
  for (void* p : c->wo) dfree(p);
  for (void* p : c->wgu) dfree(p);
  for (void* p : c->wd) dfree(p);
  for (float* p : c->g_attn) dfree(p);
  for (float* p : c->g_mlp) dfree(p);
  dfree(c->g_final);
  for (auto& kv : c->readout) {
    dfree(kv.second.first);
    dfree(kv.second.second);
  }
  dfree(c->d_layers); dfree(c->kpool); dfree(c->vpool); dfree(c->d_block_table); dfree(c->d_hist);
  if (c->h_block_table) (void)hipHostFree(c->h_block_table);
  dfree(c->d_cos); dfree(c->d_sin);
  dfree(c->d_tw);
  dfree(c->d_x); dfree(c->d_head_part); dfree(c->d_counters); dfree(c->d_ctl);
  dfree(c->d_ring_tok); dfree(c->d_ring_exit); dfree(c->d_ring_would); dfree(c->d_ring_conf); dfree(c->d_ring_mass);
  dfree(c->d_force_tok); dfree(c->d_force_exit); dfree(c->d_dbg_r); dfree(c->d_dbg_f);
  dfree(c->d_timeline);
  dfree(c->bbuf.X); dfree(c->bbuf.Q); dfree(c->bbuf.O); dfree(c->bbuf.Act);
  dfree(c->bbuf.gemm_ws); dfree(c->bbuf.attn_ws); dfree(c->bbuf.tile_ctr);
  if (c->ev0) (void)hipEventDestroy(c->ev0);
  if (c->ev1) (void)hipEventDestroy(c->ev1);
  if (c->own_stream && c->stream) (void)hipStreamDestroy(c->stream);
  if (c->params_pinned) (void)hipHostFree(c->params_pinned);
  give_slot(c->slot);
  delete c;
}


// Every entry point runs its body under guarded(): no C++ exception
// (std::bad_alloc from a container, for instance) crosses the C ABI.
int ee_create(const ee_config* cfg, void* hip_stream, ee_ctx** out) {
  return guarded(nullptr, [&]() { return create_impl(cfg, hip_stream, out); });
}
int ee_load_weights(ee_ctx* c, const ee_tensor* tensors, int32_t n_tensors) {
  return guarded(c, [&]() { return load_weights_impl(c, tensors, n_tensors); });
}
int ee_prefill(ee_ctx* c, const int32_t* tokens, int32_t n, int32_t* out_first_token) {
  return guarded(c, [&]() { return prefill_impl(c, tokens, n, out_first_token); });
}
int ee_refresh(ee_ctx* c, int32_t n) {
  return guarded(c, [&]() { return refresh_impl(c, n); });
}
int ee_decode_n_ex(ee_ctx* c, float tau, int32_t exit_layer, int32_t n, const int32_t* force_tokens,
                   const int32_t* force_exit, int32_t* tokens, int32_t* exited, float* conf,
                   int32_t* would_exit) {
  return guarded(c, [&]() { return decode_n_ex_impl(c, tau, exit_layer, n, force_tokens, force_exit, tokens, exited, conf, would_exit); });
}
int ee_decode_n(ee_ctx* c, float tau, int32_t exit_layer, int32_t n, int32_t* tokens,
                int32_t* exited, float* conf) {
  return guarded(c, [&]() { return decode_n_impl(c, tau, exit_layer, n, tokens, exited, conf); });
}
int ee_decode_n_noalloc(ee_ctx* c, float tau, int32_t exit_layer, int32_t n, int32_t* d_tokens,
                        int32_t* d_exited, float* d_conf) {
  return guarded(c, [&]() { return decode_n_noalloc_impl(c, tau, exit_layer, n, d_tokens, d_exited, d_conf); });
}
int ee_decode_step(ee_ctx* c, float tau, int32_t exit_layer, int32_t* out_token,
                   int32_t* out_exited, float* out_conf) {
  return guarded(c, [&]() { return decode_step_impl(c, tau, exit_layer, out_token, out_exited, out_conf); });
}
int ee_decode_step_ex(ee_ctx* c, float tau, int32_t exit_layer, int32_t input_token,
                      int32_t force_exit, ee_debug* dbg) {
  return guarded(c, [&]() { return decode_step_ex_impl(c, tau, exit_layer, input_token, force_exit, dbg); });
}
int ee_calibrate_threshold(ee_ctx* c, const int32_t* prompts, const int32_t* prompt_lens,
                           int32_t n_prompts, int32_t n_gen, int32_t exit_layer, int32_t mode,
                           float target, float* out_tau) {
  return guarded(c, [&]() { return calibrate_threshold_impl(c, prompts, prompt_lens, n_prompts, n_gen, exit_layer, mode, target, out_tau); });
}
int ee_calibration_record(ee_ctx* c, int32_t n, float* confs, float* masses) {
  return guarded(c, [&]() { return calibration_record_impl(c, n, confs, masses); });
}
int ee_set_readout_bias(ee_ctx* c, int32_t exit_layer, const float* b, int32_t on_device) {
  return guarded(c, [&]() { return set_readout_bias_impl(c, exit_layer, b, on_device); });
}
int ee_set_prefill_chunk(ee_ctx* c, int32_t positions) {
  return guarded(c, [&]() { return set_prefill_chunk_impl(c, positions); });
}
int ee_set_fill_policy(ee_ctx* c, int32_t policy) {
  return guarded(c, [&]() { return set_fill_policy_impl(c, policy); });
}
int ee_stream_probe(ee_ctx* c, int64_t bytes, int32_t reps, float* out_gbps) {
  return guarded(c, [&]() { return stream_probe_impl(c, bytes, reps, out_gbps); });
}
int ee_set_confidence_measure(ee_ctx* c, int32_t measure) {
  return guarded(c, [&]() { return set_confidence_measure_impl(c, measure); });
}
int ee_head_eval(ee_ctx* c, int32_t readout_layer, const float* x, int32_t* out_token,
                 float* out_conf, float* out_logits) {
  return guarded(c, [&]() { return head_eval_impl(c, readout_layer, x, out_token, out_conf, out_logits); });
}
int ee_read_kv(ee_ctx* c, int32_t layer, int32_t pos, float* k_out, float* v_out) {
  return guarded(c, [&]() { return read_kv_impl(c, layer, pos, k_out, v_out); });
}
int ee_set_persistent(ee_ctx* c, int32_t wgs_per_cu) {
  return guarded(c, [&]() { return set_persistent_impl(c, wgs_per_cu); });
}
int ee_set_persistent_grid(ee_ctx* c, int32_t nwg) {
  return guarded(c, [&]() { return set_persistent_grid_impl(c, nwg); });
}
int ee_set_timeline(ee_ctx* c, int32_t capacity) {
  return guarded(c, [&]() { return set_timeline_impl(c, capacity); });
}
int ee_read_timeline(ee_ctx* c, uint64_t* out, int32_t n) {
  return guarded(c, [&]() { return read_timeline_impl(c, out, n); });
}
int ee_last_decode_ms(ee_ctx* c, float* out_ms) {
  return guarded(c, [&]() { return last_decode_ms_impl(c, out_ms); });
}
int ee_reset(ee_ctx* c) {
  return guarded(c, [&]() { return reset_impl(c); });
}
void ee_destroy(ee_ctx* c) {
  try {
    destroy_impl(c);
  } catch (...) {
  }
}

}  // extern "C"
