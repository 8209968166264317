"""The gated decoder, one token at a time (plus a batched prompt pass).

What one decode step computes (Section 4, step five):
  1. run layers 1..L_e on the token's embedding;
  2. readout: z = W_r h + b_r, then the model's own final RMSNorm and tied
     unembedding (Section 2 "Readout, or lens"; Appendix B);
  3. confidence c = max softmax probability of those logits; exit iff c > tau
     (Section 2 "Confidence gate": the early answer is accepted when the best
     token's probability exceeds the threshold);
  4. exit: emit the readout's argmax and supply the cache entries of layers
     L_e+1..L by projecting the exit-layer state through those layers' key and
     value matrices (Section 4, step five);
     fallback: run layers L_e+1..L and emit the full model's argmax.
Decoding is greedy (Appendix B records greedy outputs).

Readings where the paper is silent:
  * exit_layer counts layers run before the readout (1..L); exit_layer 0 means
    the plain ungated model (no readout, no gate), the baseline.
  * The projected "exit-layer state" is the raw residual h_{L_e} (the readout's
    input); each skipped layer applies its own input RMSNorm gain, its W_k/W_v
    and RoPE at the token's own position.
  * The gate compares in fp32: float32(c) > float32(tau). Argmax ties go to the
    lowest token id. The reported confidence is the readout's even on fallback
    steps; for the ungated model it is the full head's.
  * Cache entries are stored rounded to the weight storage type.
  * The first generated token comes from the prompt pass at full depth,
    ungated; each decode step consumes the previous output token.
"""
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
import math
import os

import numpy as np

from .numerics import bf16_bits_to_f64, confidence_measures, head_stats, rmsnorm, rope, round_to_storage, silu


def _mat(a: np.ndarray, wdtype: str, pool=None) -> np.ndarray:
    """Exact fp64 value of a stored matrix (bf16 bit patterns or fp32)."""
    conv = bf16_bits_to_f64 if wdtype == "bf16" else (lambda x: np.asarray(x, np.float32).astype(np.float64))
    if pool is None or a.ndim != 2 or a.shape[0] < 64:
        return conv(a)
    out = np.empty(a.shape, dtype=np.float64)
    step = max(1, (1 << 21) // a.shape[1])

    def part(r):
        out[r:r + step] = conv(a[r:r + step])
    list(pool.map(part, range(0, a.shape[0], step)))
    return out


@dataclass
class StepResult:
    token: int                 # emitted token
    exited: bool               # branch taken
    conf: float                # readout confidence under the chosen measure (full head's when ungated)
    would_exit: bool           # gate decision before any forcing
    readout_token: int = -1
    gap_readout: float = math.inf
    full_token: int = -1       # full head argmax (-1 when the upper layers were skipped)
    gap_full: float = math.inf
    conf_full: float = math.nan
    h_exit: np.ndarray = None  # residual after layer L_e
    h_final: np.ndarray = None # residual after layer L (None when exited)
    logits_readout: np.ndarray = None
    logits_full: np.ndarray = None
    measures: dict = None      # all three measures of the head that set conf


class OracleDecoder:
    def __init__(self, cfg, weights: dict, max_seq: int):
        self.cfg = cfg
        wd = cfg.wdtype
        pool = ThreadPoolExecutor(min(16, len(os.sched_getaffinity(0))))
        mat = lambda a: _mat(a, wd, pool)
        self.E = mat(weights["embed"])
        self.layers = []
        for l in range(cfg.n_layers):
            p = f"layers.{l}."
            self.layers.append(dict(
                g_attn=np.asarray(weights[p + "attn_norm"], np.float64),
                wq=mat(weights[p + "wq"]), wk=mat(weights[p + "wk"]),
                wv=mat(weights[p + "wv"]), wo=mat(weights[p + "wo"]),
                g_mlp=np.asarray(weights[p + "mlp_norm"], np.float64),
                wg=mat(weights[p + "w_gate"]), wu=mat(weights[p + "w_up"]),
                wd=mat(weights[p + "w_down"])))
        self.g_final = np.asarray(weights["final_norm"], np.float64)
        self.readouts = {}
        for L in cfg.readout_layers:
            self.readouts[L] = (mat(weights[f"readout.{L}.w"]),
                                np.asarray(weights[f"readout.{L}.b"], np.float64))
        pool.shutdown()
        self.max_seq = max_seq
        shape = (cfg.n_layers, max_seq, cfg.n_kv_heads, cfg.head_dim)
        self.kcache = np.zeros(shape)
        self.vcache = np.zeros(shape)
        self.hist = np.full(max_seq, -1, dtype=np.int64)  # input token of every position
        self.pos = 0

    # -- bookkeeping -------------------------------------------------------
    def reset(self):
        self.kcache[:] = 0.0
        self.vcache[:] = 0.0
        self.hist[:] = -1
        self.pos = 0

    def _store(self, l, t, k, v):
        self.kcache[l, t] = round_to_storage(k, self.cfg.wdtype)
        self.vcache[l, t] = round_to_storage(v, self.cfg.wdtype)

    # -- one layer for one token ------------------------------------------
    def _kv_proj(self, l, a, t):
        c = self.cfg
        lw = self.layers[l]
        k = rope((lw["wk"] @ a).reshape(c.n_kv_heads, c.head_dim), t, c.rope_base)
        v = (lw["wv"] @ a).reshape(c.n_kv_heads, c.head_dim)
        return k, v

    def attend(self, q, kc, vc):
        """q [A, D]; kc, vc [T, K, D] -> o [A, D]. Query head i reads KV head
        i // (A/K); every position up to and including the current one."""
        c = self.cfg
        group = c.n_q_heads // c.n_kv_heads
        o = np.empty_like(q)
        for i in range(c.n_q_heads):
            g = i // group
            s = kc[:, g, :] @ q[i] / math.sqrt(c.head_dim)
            p = np.exp(s - s.max())
            p /= p.sum()
            o[i] = p @ vc[:, g, :]
        return o

    def layer(self, l, h, t):
        c = self.cfg
        lw = self.layers[l]
        a = rmsnorm(h, lw["g_attn"], c.rms_eps)
        q = rope((lw["wq"] @ a).reshape(c.n_q_heads, c.head_dim), t, c.rope_base)
        k, v = self._kv_proj(l, a, t)
        self._store(l, t, k, v)
        o = self.attend(q, self.kcache[l, :t + 1], self.vcache[l, :t + 1])
        h = h + lw["wo"] @ o.reshape(-1)
        m = rmsnorm(h, lw["g_mlp"], c.rms_eps)
        return h + lw["wd"] @ (silu(lw["wg"] @ m) * (lw["wu"] @ m))

    def fill(self, l, h_exit, t):
        """Cache entry of a skipped layer: the exit-layer state projected
        through layer l's key and value matrices (Section 4, step five)."""
        a = rmsnorm(h_exit, self.layers[l]["g_attn"], self.cfg.rms_eps)
        k, v = self._kv_proj(l, a, t)
        self._store(l, t, k, v)

    # -- heads ---------------------------------------------------------------
    def full_logits(self, h):
        return self.E @ rmsnorm(h, self.g_final, self.cfg.rms_eps)

    def readout_logits(self, h_exit, exit_layer):
        W, b = self.readouts[exit_layer]
        z = W @ h_exit + b
        return self.E @ rmsnorm(z, self.g_final, self.cfg.rms_eps)

    # -- decode ----------------------------------------------------------------
    def decode_step(self, token: int, tau: float, exit_layer: int, force_exit: int = -1,
                    keep_logits: bool = False, measure: str = "maxprob") -> StepResult:
        """One gated step. measure selects the confidence the gate compares
        with tau (maxprob, margin or negentropy); exit iff it exceeds tau."""
        c = self.cfg
        L = c.n_layers
        if not (0 <= exit_layer <= L):
            raise ValueError("exit_layer out of range")
        if exit_layer and exit_layer not in self.readouts:
            raise ValueError(f"no readout at layer {exit_layer}")
        if math.isnan(tau):
            raise ValueError("tau is NaN")
        t = self.pos
        if t >= self.max_seq:
            raise ValueError("cache capacity exceeded")
        self.hist[t] = token
        h = self.E[token].copy()
        for l in range(exit_layer):
            h = self.layer(l, h, t)
        h_exit = h.copy()
        res = StepResult(token=-1, exited=False, conf=math.nan, would_exit=False, h_exit=h_exit)
        if exit_layer:
            lr = self.readout_logits(h_exit, exit_layer)
            res.readout_token, res.conf, res.gap_readout = head_stats(lr)
            res.measures = confidence_measures(lr)
            res.conf = res.measures[measure]
            res.would_exit = bool(np.float32(res.conf) > np.float32(tau))
            res.exited = res.would_exit if force_exit < 0 else bool(force_exit)
            if keep_logits:
                res.logits_readout = lr
        if res.exited:
            for l in range(exit_layer, L):
                self.fill(l, h_exit, t)
            res.token = res.readout_token
        else:
            for l in range(exit_layer, L):
                h = self.layer(l, h, t)
            lf = self.full_logits(h)
            res.full_token, res.conf_full, res.gap_full = head_stats(lf)
            res.token = res.full_token
            res.h_final = h
            if not exit_layer:
                res.measures = confidence_measures(lf)
                res.conf_full = res.measures[measure]
                res.conf = res.conf_full
            if keep_logits:
                res.logits_full = lf
        self.pos = t + 1
        return res

    def prefill(self, tokens, progress=None) -> int:
        """Prompt pass at full depth over positions pos..pos+P-1, all layers,
        batched over positions with a causal mask. Returns the first generated
        token (argmax of the full head at the last prompt position).
        progress, if given, is called with each layer index once it is done."""
        c = self.cfg
        tokens = np.asarray(tokens, dtype=np.int64)
        P = tokens.size
        t0 = self.pos
        if P == 0:
            raise ValueError("empty prompt")
        if t0 + P > self.max_seq:
            raise ValueError("cache capacity exceeded")
        T = t0 + P
        self.hist[t0:T] = tokens
        pos = np.arange(t0, T)
        group = c.n_q_heads // c.n_kv_heads
        H = self.E[tokens].copy()
        for l, lw in enumerate(self.layers):
            a = rmsnorm(H, lw["g_attn"], c.rms_eps)
            q = rope((a @ lw["wq"].T).reshape(P, c.n_q_heads, c.head_dim), pos, c.rope_base)
            k = rope((a @ lw["wk"].T).reshape(P, c.n_kv_heads, c.head_dim), pos, c.rope_base)
            v = (a @ lw["wv"].T).reshape(P, c.n_kv_heads, c.head_dim)
            self.kcache[l, t0:T] = round_to_storage(k, c.wdtype)
            self.vcache[l, t0:T] = round_to_storage(v, c.wdtype)
            kc, vc = self.kcache[l, :T], self.vcache[l, :T]
            o = np.empty((P, c.n_q_heads, c.head_dim))
            mask = np.arange(T)[None, :] > pos[:, None]
            for i in range(c.n_q_heads):
                g = i // group
                s = q[:, i, :] @ kc[:, g, :].T / math.sqrt(c.head_dim)
                s[mask] = -np.inf
                p = np.exp(s - s.max(axis=1, keepdims=True))
                p /= p.sum(axis=1, keepdims=True)
                o[:, i, :] = p @ vc[:, g, :]
            H = H + o.reshape(P, -1) @ lw["wo"].T
            m = rmsnorm(H, lw["g_mlp"], c.rms_eps)
            H = H + (silu(m @ lw["wg"].T) * (m @ lw["wu"].T)) @ lw["wd"].T
            if progress is not None:
                progress(l)
        self.pos = T
        self.last_prefill_stats = head_stats(self.full_logits(H[-1]))  # (token, conf, gap)
        return self.last_prefill_stats[0]

    def refresh(self, n: int) -> None:
        """Full-depth pass over the n most recent positions with their own
        input tokens: their cache entries at every layer are recomputed
        exactly, replacing the entries the KV-absence fill projected for
        exited tokens (Section 11: a periodic full-depth pass over the most
        recent tokens recovers the drift of the reconstructed cache). The
        position and the next input are unchanged."""
        if not (1 <= n <= self.pos):
            raise ValueError("refresh needs 1 <= n <= position")
        end = self.pos
        toks = self.hist[end - n:end].copy()
        self.pos = end - n
        self.prefill(toks)
        assert self.pos == end

    def generate(self, first_token: int, tau: float, exit_layer: int, n: int,
                 force_tokens=None, force_exit=None, keep_logits=False, measure="maxprob"):
        """n decode steps. Free-running unless force_tokens (input token per
        step) is given; force_exit (per step, -1/0/1) imposes branches."""
        out = []
        tok = first_token
        for i in range(n):
            if force_tokens is not None:
                tok = int(force_tokens[i])
            fe = -1 if force_exit is None else int(force_exit[i])
            r = self.decode_step(tok, tau, exit_layer, fe, keep_logits, measure)
            out.append(r)
            tok = r.token
        return out
