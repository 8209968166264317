"""Pins of the oracle's elementary operations against library routines,
closed forms and brute force (CPU only)."""
import math

import numpy as np
import pytest
import torch

from oracle.numerics import bf16_bits_to_f64, confidence_measures, head_stats, rmsnorm, rope, round_to_storage, silu
import synth


def test_bf16_rounding_matches_torch_on_fp32_values():
    rng = np.random.default_rng(3)
    x32 = (rng.standard_normal(200_000) * np.exp(rng.uniform(-20, 20, 200_000))).astype(np.float32)
    # values exactly half-way between two bf16 numbers exercise ties-to-even
    base = (rng.integers(0, 1 << 15, 1000).astype(np.uint32) << 16) | 0x8000
    x32 = np.concatenate([x32, base.view(np.float32)])
    x32 = x32[np.isfinite(x32)]
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_to_storage(x32.astype(np.float64), "bf16"), ref)


def test_bf16_rounding_special_cases():
    eps = 2.0 ** -7                     # bf16 spacing in [1, 2)
    assert round_to_storage(np.array([1 + eps / 2]), "bf16")[0] == 1.0            # tie -> even
    assert round_to_storage(np.array([1 + 3 * eps / 2]), "bf16")[0] == 1 + 2 * eps  # tie -> even (up)
    assert round_to_storage(np.array([1 + eps / 2 + 1e-12]), "bf16")[0] == 1 + eps
    assert round_to_storage(np.array([-(2 - eps / 4)]), "bf16")[0] == -2.0        # carry into exponent
    assert round_to_storage(np.array([0.0]), "bf16")[0] == 0.0


def test_generator_bf16_bits_match_torch_and_decode_exactly():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(10_000).astype(np.float32)
    bits = synth.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bits, ref)
    np.testing.assert_array_equal(bf16_bits_to_f64(bits),
                                  torch.from_numpy(x).to(torch.bfloat16).double().numpy())


def test_rmsnorm_library_and_closed_form():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((7, 96))
    g = rng.uniform(0.5, 2, 96)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-6)
    np.testing.assert_allclose(rmsnorm(x, g, 1e-6), ref.numpy(), rtol=1e-13, atol=0)
    c = -3.0
    y = rmsnorm(np.full(8, c), np.full(8, 2.0), 1e-6)
    np.testing.assert_allclose(y, 2.0 * c / math.sqrt(c * c + 1e-6), rtol=1e-15)


def test_rope_matches_transformers_rotate_half():
    from transformers.models.qwen2.modeling_qwen2 import apply_rotary_pos_emb
    rng = np.random.default_rng(6)
    D, base = 64, 10000.0
    q = rng.standard_normal((5, 3, D))           # positions x heads x D
    k = rng.standard_normal((5, 2, D))
    pos = np.array([0, 1, 17, 513, 9215])
    inv = 1.0 / (base ** (np.arange(0, D, 2, dtype=np.float64) / D))
    ang = pos[:, None] * inv[None, :]
    emb = np.concatenate([ang, ang], axis=-1)
    cos = torch.from_numpy(np.cos(emb))[None]    # [1, P, D]
    sin = torch.from_numpy(np.sin(emb))[None]
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]  # [1, heads, P, D]
    kt = torch.from_numpy(k).permute(1, 0, 2)[None]
    qr, kr = apply_rotary_pos_emb(qt, kt, cos, sin)
    np.testing.assert_allclose(rope(q, pos, base), qr[0].permute(1, 0, 2).numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(rope(k, pos, base), kr[0].permute(1, 0, 2).numpy(), rtol=1e-10, atol=1e-10)


def test_rope_invariants():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((1, 128))
    k = rng.standard_normal((1, 128))
    np.testing.assert_array_equal(rope(q, 0, 1e4), q)                       # position 0 = identity
    np.testing.assert_allclose(np.linalg.norm(rope(q, 77, 1e4)), np.linalg.norm(q), rtol=1e-13)
    d1 = float(rope(q, 300, 1e4)[0] @ rope(k, 290, 1e4)[0])                # relative position only
    d2 = float(rope(q, 12, 1e4)[0] @ rope(k, 2, 1e4)[0])
    assert abs(d1 - d2) < 1e-10


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(),
                               rtol=1e-14, atol=1e-300)


def test_head_stats_brute_force():
    from scipy.special import softmax
    rng = np.random.default_rng(8)
    for trial in range(20):
        V = int(rng.integers(2, 5000))
        lg = rng.standard_normal(V) * rng.uniform(0.1, 10)
        if trial % 3 == 0:                       # planted tie at the max: lowest index wins
            i, j = sorted(rng.choice(V, 2, replace=False))
            lg[i] = lg[j] = lg.max() + 1.0
        j, conf, gap = head_stats(lg)
        order = sorted(range(V), key=lambda t: (-lg[t], t))   # brute-force ranking
        assert j == order[0]
        assert abs(conf - softmax(lg).max()) < 1e-12
        assert gap == lg[order[0]] - lg[order[1]]
    j, conf, gap = head_stats(np.zeros(4096))
    assert j == 0 and conf == 1.0 / 4096 and gap == 0.0


def test_confidence_measures_library_and_closed_forms():
    """The three confidence measures (Section 10) against library routines and
    closed forms: negative entropy vs scipy's entropy, the best probability
    vs the head's own confidence, margins and entropies of two-token and
    uniform distributions, and ties."""
    from scipy.special import softmax
    from scipy.stats import entropy
    rng = np.random.default_rng(11)
    for V, scale in ((2, 1.0), (7, 3.0), (1000, 5.0), (151936, 5.0)):
        x = rng.standard_normal(V) * scale
        m = confidence_measures(x)
        p = softmax(x)
        assert m["maxprob"] == pytest.approx(head_stats(x)[1], rel=1e-12)
        assert m["negentropy"] == pytest.approx(-entropy(p), rel=1e-10, abs=1e-12)
        q = np.sort(p)
        assert m["margin"] == pytest.approx(q[-1] - q[-2], rel=1e-10, abs=1e-15)
        assert 0.0 <= m["margin"] <= m["maxprob"] <= 1.0
        assert -math.log(V) - 1e-9 <= m["negentropy"] <= 0.0
    # two tokens, logit difference d: p = sigmoid(d)
    for d in (0.0, 0.3, 2.0, 9.0):
        m = confidence_measures(np.array([d, 0.0]))
        s = 1.0 / (1.0 + math.exp(-d))
        assert m["margin"] == pytest.approx(math.tanh(d / 2), abs=1e-14)
        assert m["negentropy"] == pytest.approx(s * math.log(s) + (1 - s) * math.log(1 - s), abs=1e-14)
    # uniform: no margin, entropy log V
    m = confidence_measures(np.full(4096, 1.25))
    assert m["margin"] == 0.0 and m["maxprob"] == pytest.approx(1 / 4096)
    assert m["negentropy"] == pytest.approx(-math.log(4096), rel=1e-13)
    # a tie at the top: zero margin whatever the rest
    x = rng.standard_normal(500)
    x[[17, 300]] = x.max() + 1.0
    assert confidence_measures(x)["margin"] == 0.0
    # a dominant token: maxprob and margin near 1, entropy near 0 (underflow safe)
    x = np.zeros(1000)
    x[5] = 800.0
    m = confidence_measures(x)
    assert m["maxprob"] == 1.0 and m["margin"] == 1.0 and m["negentropy"] == 0.0
