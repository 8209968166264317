"""Pins of the oracle's decoder, gate, readout, KV fill and calibration.

Independent references: transformers' Qwen2 decoder in fp64 (a library
implementation of the same pre-norm GQA/RoPE/SwiGLU decoder), brute force,
closed forms and invariants of the gate."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from oracle.numerics import round_to_storage
from tests.conftest import weights_for
from tests.hf_ref import build_qwen2

CFG = synth.get_config("tiny")
P = 16


def rel(a, b):
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b)) / np.linalg.norm(np.asarray(b)))


@pytest.fixture(scope="module")
def w():
    return weights_for("tiny")


@pytest.fixture(scope="module")
def hf(w):
    return build_qwen2(CFG, w)


def seq(n, seed=11):
    return synth.prompts(CFG, seed, n)


def test_full_forward_matches_transformers(w, hf):
    toks = seq(40)
    o = oracle.OracleDecoder(CFG, w, 64)
    ours = [o.decode_step(int(t), math.inf, 0, keep_logits=True).logits_full for t in toks]
    with torch.no_grad():
        ref = hf(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].numpy()
    for i in range(len(toks)):
        assert rel(ours[i], ref[i]) < 1e-6, i
        assert int(np.argmax(ours[i])) == int(np.argmax(ref[i]))


def test_prefill_equals_sequential_decode(w):
    p = seq(P, 1)
    a = oracle.OracleDecoder(CFG, w, 64)
    g0 = a.prefill(p)
    b = oracle.OracleDecoder(CFG, w, 64)
    rs = [b.decode_step(int(t), math.inf, 0) for t in p]
    assert g0 == rs[-1].token
    np.testing.assert_allclose(a.kcache[:, :P], b.kcache[:, :P], rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(a.vcache[:, :P], b.vcache[:, :P], rtol=1e-6, atol=1e-9)
    assert a.pos == b.pos == P


def test_gated_infinite_tau_is_bit_identical_to_ungated(w):
    p = seq(P, 1)
    a = oracle.OracleDecoder(CFG, w, 64)
    b = oracle.OracleDecoder(CFG, w, 64)
    ra = a.generate(a.prefill(p), math.inf, 2, 24)
    rb = b.generate(b.prefill(p), math.inf, 0, 24)
    assert [r.token for r in ra] == [r.token for r in rb]
    assert not any(r.exited for r in ra)
    for x, y in zip(ra, rb):
        np.testing.assert_array_equal(x.h_final, y.h_final)
    np.testing.assert_array_equal(a.kcache, b.kcache)


@pytest.mark.parametrize("tau,expect", [(1.0, 0), (2.0, 0), (0.0, 24), (-1.0, 24), (-math.inf, 24)])
def test_gate_limits(w, tau, expect):
    o = oracle.OracleDecoder(CFG, w, 64)
    rs = o.generate(o.prefill(seq(P, 1)), tau, 2, 24, force_tokens=seq(24, 5))
    assert sum(r.exited for r in rs) == expect
    for r in rs:
        assert 1.0 / CFG.vocab <= r.conf <= 1.0


def test_teacher_forced_confidence_independent_of_tau_and_exits_monotone(w):
    toks = seq(32, 5)
    runs = {}
    for tau in (math.inf, 0.9, 0.7, 0.5, 0.3, 0.0):
        o = oracle.OracleDecoder(CFG, w, 64)
        runs[tau] = o.generate(o.prefill(seq(P, 1)), tau, 2, 32, force_tokens=toks)
    base = [r.conf for r in runs[math.inf]]
    prev = set()
    for tau in (math.inf, 0.9, 0.7, 0.5, 0.3, 0.0):
        assert [r.conf for r in runs[tau]] == base         # layers <= L_e never read filled KV
        ex = {i for i, r in enumerate(runs[tau]) if r.exited}
        assert ex == {i for i, c in enumerate(base) if np.float32(c) > np.float32(tau)}
        assert prev <= ex
        prev = ex
    assert 0 < len({i for i, r in enumerate(runs[0.5]) if r.exited}) < 32


@pytest.mark.parametrize("measure,never,always", [("margin", 1.0, -1e-30), ("negentropy", 0.0, -math.inf)])
def test_gate_measures(w, measure, never, always):
    """The gate under the margin and negative-entropy measures (Section 10):
    the measure's range fixes the thresholds that never / always exit, the
    gated step's conf is the measure of the readout's logits, and max-prob
    mode is the default."""
    toks = seq(24, 5)
    o = oracle.OracleDecoder(CFG, w, 64)
    rs = o.generate(o.prefill(seq(P, 1)), math.inf, 2, 24, force_tokens=toks, keep_logits=True,
                    measure=measure)
    for r in rs:
        assert r.conf == oracle.confidence_measures(r.logits_readout)[measure]
    for tau, expect in ((never, 0), (always, 24)):
        o = oracle.OracleDecoder(CFG, w, 64)
        rs2 = o.generate(o.prefill(seq(P, 1)), tau, 2, 24, force_tokens=toks, measure=measure)
        assert sum(r.exited for r in rs2) == expect
        assert [r.conf for r in rs2] == [r.conf for r in rs]
    o = oracle.OracleDecoder(CFG, w, 64)
    d = o.generate(o.prefill(seq(P, 1)), 0.5, 2, 24, force_tokens=toks)
    o = oracle.OracleDecoder(CFG, w, 64)
    m = o.generate(o.prefill(seq(P, 1)), 0.5, 2, 24, force_tokens=toks, measure="maxprob")
    assert [(r.token, r.exited, r.conf) for r in d] == [(r.token, r.exited, r.conf) for r in m]


def test_readout_special_cases(w):
    """Logit lens (W = I, b = 0) at L_e = L equals the full head; a permutation
    readout permutes the residual; an offset of -h zeroes the normalised state,
    giving uniform probabilities (conf = 1/V, token 0)."""
    L, H = CFG.n_layers, CFG.hidden
    cfg = CFG.with_readouts((L,))
    w2 = dict(w)
    w2[f"readout.{L}.w"] = np.eye(H, dtype=np.float32)
    w2[f"readout.{L}.b"] = np.zeros(H, np.float32)
    o = oracle.OracleDecoder(cfg, w2, 64)
    o.prefill(seq(P, 1))
    r = o.decode_step(7, math.inf, L, keep_logits=True)
    np.testing.assert_array_equal(r.logits_readout, r.logits_full)
    assert r.readout_token == r.full_token and r.conf == r.conf_full

    perm = np.random.default_rng(9).permutation(H)
    Pm = np.zeros((H, H), np.float32)
    Pm[np.arange(H), perm] = 1.0                  # (Pm h)[i] = h[perm[i]]
    w2[f"readout.{L}.w"] = Pm
    o = oracle.OracleDecoder(cfg, w2, 64)
    o.prefill(seq(P, 1))
    r = o.decode_step(7, math.inf, L, keep_logits=True)
    ref = o.E @ oracle.rmsnorm(r.h_final[perm], o.g_final, CFG.rms_eps)
    np.testing.assert_allclose(r.logits_readout, ref, rtol=1e-12, atol=1e-12)

    cfg2 = CFG.with_readouts((2,))
    w3 = dict(w)
    w3["readout.2.w"] = np.zeros((H, H), np.float32)
    w3["readout.2.b"] = np.zeros(H, np.float32)
    o = oracle.OracleDecoder(cfg2, w3, 64)
    o.prefill(seq(P, 1))
    r = o.decode_step(7, 0.5, 2, keep_logits=True)       # z = 0: every logit is 0
    assert r.conf == 1.0 / CFG.vocab and r.readout_token == 0 and not r.exited
    k, beta = 37, 3.0
    w3["readout.2.b"] = np.zeros(H, np.float32)
    w3["readout.2.b"][k] = beta                          # z = beta e_k
    o = oracle.OracleDecoder(cfg2, w3, 64)
    o.prefill(seq(P, 1))
    r = o.decode_step(7, 0.5, 2, keep_logits=True)
    scale = beta / math.sqrt(beta * beta / H + CFG.rms_eps) * CFG.final_norm_gain
    np.testing.assert_allclose(r.logits_readout, o.E[:, k] * scale, rtol=1e-12)
    assert r.readout_token == int(np.argmax(o.E[:, k]))


def test_readout_argmax_and_conf_brute_force(w):
    from scipy.special import softmax
    o = oracle.OracleDecoder(CFG, w, 64)
    o.prefill(seq(P, 1))
    for t in seq(8, 21):
        r = o.decode_step(int(t), math.inf, 2, keep_logits=True)
        lg = r.logits_readout
        order = np.lexsort((np.arange(lg.size), -lg))
        assert r.readout_token == order[0]
        assert abs(r.conf - softmax(lg).max()) < 1e-12
        assert r.gap_readout == lg[order[0]] - lg[order[1]]


def test_kv_fill_matches_transformers_projection(w, hf):
    from transformers.models.qwen2.modeling_qwen2 import apply_rotary_pos_emb
    o = oracle.OracleDecoder(CFG, w, 64)
    o.prefill(seq(P, 1))
    t = o.pos
    r = o.decode_step(123, -1.0, 2)                   # tau < 0 always exits
    assert r.exited
    h = torch.from_numpy(r.h_exit)[None, None]        # [1, 1, H]
    pos_ids = torch.tensor([[t]])
    with torch.no_grad():
        cos, sin = hf.model.rotary_emb(h, pos_ids)
        for l in range(2, CFG.n_layers):
            lay = hf.model.layers[l]
            a = lay.input_layernorm(h)
            k = lay.self_attn.k_proj(a).view(1, 1, CFG.n_kv_heads, CFG.head_dim).transpose(1, 2)
            v = lay.self_attn.v_proj(a).view(1, 1, CFG.n_kv_heads, CFG.head_dim).transpose(1, 2)
            k, _ = apply_rotary_pos_emb(k, k, cos, sin)
            np.testing.assert_allclose(o.kcache[l, t], k[0, :, 0].numpy(), rtol=1e-6, atol=1e-7)
            np.testing.assert_allclose(o.vcache[l, t], v[0, :, 0].numpy(), rtol=1e-6, atol=1e-7)


def test_steps_after_exit_attend_to_filled_entries(w, hf):
    """After exits, a full-depth step uses the cache as filled: transformers,
    given the oracle's cache (with the filled entries) as its past, must
    produce the same logits for the next token."""
    from transformers import DynamicCache
    o = oracle.OracleDecoder(CFG, w, 64)
    o.prefill(seq(P, 1))
    o.generate(5, 0.0, 2, 3, force_tokens=[5, 6, 7], force_exit=[1, 1, 1])
    T = o.pos
    r = o.decode_step(9, math.inf, 0, keep_logits=True)
    cache = DynamicCache(config=hf.config)
    for l in range(CFG.n_layers):
        k = torch.from_numpy(o.kcache[l, :T]).permute(1, 0, 2)[None].contiguous()
        v = torch.from_numpy(o.vcache[l, :T]).permute(1, 0, 2)[None].contiguous()
        cache.update(k, v, l)
    with torch.no_grad():
        out = hf(torch.tensor([[9]]), past_key_values=cache, position_ids=torch.tensor([[T]]),
                 use_cache=True)
    assert rel(r.logits_full, out.logits[0, 0].numpy()) < 1e-6


def test_calibration_exit_rate_replay(w):
    """Calibrate on a full-depth run, replay the same tokens: exactly k exits."""
    o = oracle.OracleDecoder(CFG, w, 64)
    toks = seq(40, 31)
    rs = o.generate(o.prefill(seq(P, 1)), math.inf, 2, 40, force_tokens=toks)
    confs = [np.float32(r.conf) for r in rs]
    assert len(set(confs)) == len(confs)
    for rate in (0.0, 0.1, 0.5, 0.9, 1.0):
        tau = oracle.tau_for_exit_rate(confs, rate)
        k = int(math.floor(rate * 40 + 0.5))
        o2 = oracle.OracleDecoder(CFG, w, 64)
        rr = o2.generate(o2.prefill(seq(P, 1)), tau, 2, 40, force_tokens=toks)
        assert sum(r.exited for r in rr) == k
    tau = oracle.tau_median(confs)
    assert sum(np.float32(c) > np.float32(tau) for c in confs) == 20


def test_nucleus_acceptance_brute_force():
    rng = np.random.default_rng(12)
    for _ in range(30):
        V = int(rng.integers(2, 60))
        lg = rng.standard_normal(V) * 3
        if V > 3:
            lg[1] = lg[2]
        p = np.exp(lg - lg.max()); p /= p.sum()
        order = sorted(range(V), key=lambda t: (-p[t], t))
        nucleus, mass = [], 0.0
        for t in order:                       # shortest prefix reaching 0.9
            nucleus.append(t)
            mass += p[t]
            if mass >= 0.9:
                break
        for j in range(V):
            assert oracle.nucleus_acceptable(lg, j) == (j in nucleus), (V, j)
            ahead = sum(p[t] for t in order[:order.index(j)])
            assert oracle.nucleus_mass_ahead(lg, j) == pytest.approx(ahead, abs=1e-12)


def test_tau_nucleus_grid():
    confs = np.array([0.05, 0.2, 0.35, 0.5, 0.65, 0.8, 0.95])
    ok = np.array([0, 0, 1, 1, 1, 1, 1], bool)
    # early set at tau=0.2 is {0.35..0.95}: all acceptable; at tau=0.05..0.19 one of 6 fails (5/6 < .9)
    assert oracle.tau_nucleus(confs, ok) == pytest.approx(0.2)
    assert oracle.tau_nucleus(confs, np.zeros(7, bool)) == math.inf


def test_refresh_restores_the_full_depth_cache(w):
    """A full-depth pass over every decoded position (Section 11's periodic
    refresh) replaces the projected entries of exited tokens with the cache
    an ungated run over the same tokens writes; the next step then matches
    the ungated model's."""
    toks = seq(12, 5)
    a = oracle.OracleDecoder(CFG, w, 64)
    a.prefill(seq(P, 1))
    ra = a.generate(None, 0.0, 2, 12, force_tokens=toks)        # every step exits
    assert all(r.exited for r in ra)
    b = oracle.OracleDecoder(CFG, w, 64)
    b.prefill(seq(P, 1))
    b.generate(None, 0.5, 0, 12, force_tokens=toks)              # ungated, full depth
    up = slice(2, CFG.n_layers)
    span = slice(P, P + 12)
    assert rel(a.kcache[up, span], b.kcache[up, span]) > 1e-2    # projected entries differ
    np.testing.assert_array_equal(a.hist[:P + 12], b.hist[:P + 12])
    a.refresh(12)
    assert a.pos == P + 12
    assert rel(a.kcache[:, :P + 12], b.kcache[:, :P + 12]) < 1e-12
    assert rel(a.vcache[:, :P + 12], b.vcache[:, :P + 12]) < 1e-12
    na = a.decode_step(int(toks[0]), 0.5, 0)
    nb = b.decode_step(int(toks[0]), 0.5, 0)
    assert na.token == nb.token and rel(na.h_final, nb.h_final) < 1e-12
    with pytest.raises(ValueError):
        a.refresh(0)
    with pytest.raises(ValueError):
        a.refresh(a.pos + 1)
