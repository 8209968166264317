"""GPU parity: the HIP decode path (through the C ABI) against the CPU oracle
on identical seeded inputs. See tests/gpu_helpers.py for the comparison rule."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests.conftest import weights_for
from tests.gpu_helpers import (MARGIN, check_kv, check_nucleus_mass, compare_step, engine, lockstep,
                               oracle_for, rel, worst)

pytestmark = pytest.mark.gpu

TINY_P = 16
TINY_N = 32


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


_TAU = {}


def _progress(what):
    def cb(layer):
        print(f"{what}: layer {layer} done", flush=True)
    return cb


def tiny_tau(name):
    """Median readout confidence of an oracle calibration run: 8 seeded
    prompts (seeds 100..107) of 16 tokens, 32 full-depth steps each."""
    if name not in _TAU:
        cfg = synth.get_config(name)
        confs = []
        for seed in range(100, 108):
            o = oracle_for(name, TINY_P + TINY_N)
            g = o.prefill(synth.prompts(cfg, seed, TINY_P))
            confs += [r.conf for r in o.generate(g, math.inf, 2, TINY_N)]
        _TAU[name] = oracle.tau_median(confs)
    return _TAU[name]


@pytest.mark.parametrize("persistent", [True, False], ids=["persistent", "per_op"])
@pytest.mark.parametrize("name", ["tiny", "tiny_bf16"])
def test_tiny_lockstep(name, persistent):
    cfg = synth.get_config(name)
    tau = tiny_tau(name)
    prompt = synth.prompts(cfg, 1, TINY_P)
    o = oracle_for(name, 128)
    e = engine(name, 128, persistent)
    g0 = o.prefill(prompt)
    g0_gpu = e.ee_prefill(prompt)
    if o.last_prefill_stats[2] > MARGIN:
        assert g0_gpu == g0
    rep, outside = lockstep(e, o, g0, tau, 2, TINY_N)
    # teacher-forced continuation with varied inputs
    toks = synth.prompts(cfg, 5, TINY_N)
    rep2, outside2 = lockstep(e, o, None, tau, 2, TINY_N, force_tokens=toks)
    assert outside + outside2 >= 2 * TINY_N - 4
    print(f"{name} persistent={persistent} tau={tau:.4f}", worst(rep + rep2))


@pytest.mark.parametrize("name", ["tiny", "tiny_bf16"])
def test_tiny_both_branches_exercised(name):
    cfg = synth.get_config(name)
    tau = tiny_tau(name)
    o = oracle_for(name, 128)
    g0 = o.prefill(synth.prompts(cfg, 1, TINY_P))
    rs = o.generate(g0, tau, 2, TINY_N, force_tokens=synth.prompts(cfg, 5, TINY_N))
    n_exit = sum(r.exited for r in rs)
    assert 0 < n_exit < TINY_N


@pytest.mark.parametrize("persistent", [True, False], ids=["persistent", "per_op"])
def test_tiny_decode_n_imposed_and_gated(persistent):
    """n steps in one call (the timed entry point) with teacher-forced inputs;
    first with the gate's own decisions, then with imposed exits."""
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    tau = tiny_tau(name)
    prompt = synth.prompts(cfg, 1, TINY_P)
    toks = synth.prompts(cfg, 6, TINY_N)
    for fe in (None, (np.arange(TINY_N) % 3 == 0).astype(np.int32)):
        o = oracle_for(name, 128)
        o.prefill(prompt)
        rs = o.generate(None, tau, 2, TINY_N, force_tokens=toks, force_exit=fe)
        e = engine(name, 128, persistent)
        e.ee_prefill(prompt)
        tok, ex, conf, would = e.ee_decode_n_ex(tau, 2, TINY_N, force_tokens=toks, force_exit=fe)
        for i, r in enumerate(rs):
            assert abs(conf[i] - r.conf) <= 1e-4 + 1e-3 * r.conf
            if abs(r.conf - tau) > MARGIN:
                assert would[i] == r.would_exit
                if fe is None:
                    assert ex[i] == r.exited
            if fe is not None:
                assert ex[i] == bool(fe[i])
            gap = r.gap_readout if r.exited else r.gap_full
            if gap > MARGIN and ex[i] == r.exited:
                assert tok[i] == r.token, i
        assert e.ee_position() == TINY_P + TINY_N


def measure_tol(measure, r):
    """Allowed |device - oracle| for a step's confidence: the head's logits
    carry fp32 errors of about 1e-4 relative (the max-prob bound below);
    the margin inherits them through both probabilities, the negative
    entropy through every log-probability (one per unit of entropy)."""
    c = r.measures["maxprob"]
    if measure == "maxprob":
        return 1e-4 + 1e-3 * c
    if measure == "margin":
        return 1e-4 + 2e-3 * c
    return 1e-3 * (1.0 + abs(r.conf))


@pytest.mark.parametrize("persistent", [True, False], ids=["persistent", "per_op"])
@pytest.mark.parametrize("measure", ["maxprob", "margin", "negentropy"])
def test_tiny_confidence_measures(measure, persistent):
    """The gate under each softmax confidence measure of Section 10, teacher
    forced in one call: per-step confidence against the oracle's measure of
    the readout distribution, decisions away from tau, and median
    calibration on the device against the oracle's."""
    from paper_2609_14144_amd import EE_CAL_MEDIAN
    code = {"maxprob": 0, "margin": 1, "negentropy": 2}[measure]
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 1, TINY_P)
    toks = synth.prompts(cfg, 6, TINY_N)
    o = oracle_for(name, 128)
    o.prefill(prompt)
    ref = o.generate(None, math.inf, 2, TINY_N, force_tokens=toks, measure=measure)
    tau = oracle.tau_median([r.conf for r in ref])
    o = oracle_for(name, 128)
    o.prefill(prompt)
    rs = o.generate(None, tau, 2, TINY_N, force_tokens=toks, measure=measure)
    e = engine(name, 128, persistent)
    e.ee_set_confidence_measure(code)
    e.ee_prefill(prompt)
    tok, ex, conf, would = e.ee_decode_n_ex(tau, 2, TINY_N, force_tokens=toks)
    decided = 0
    for i, r in enumerate(rs):
        assert abs(conf[i] - r.conf) <= measure_tol(measure, r), (i, conf[i], r.conf)
        if abs(r.conf - tau) > MARGIN:
            assert would[i] == r.would_exit and ex[i] == r.exited, i
            decided += 1
        gap = r.gap_readout if r.exited else r.gap_full
        if gap > MARGIN and ex[i] == r.exited:
            assert tok[i] == r.token, i
    assert decided >= TINY_N // 2 and 0 < sum(r.exited for r in rs) < TINY_N
    prompts = [synth.prompts(cfg, s, TINY_P) for s in range(100, 104)]
    confs = []
    for p in prompts:
        o = oracle_for(name, 64)
        confs += [r.conf for r in o.generate(o.prefill(p), math.inf, 2, TINY_N, measure=measure)]
    e2 = engine(name, 64, persistent)
    e2.ee_set_confidence_measure(code)
    t_gpu = e2.ee_calibrate_threshold(prompts, TINY_N, 2, EE_CAL_MEDIAN, 0.0)
    t_ref = oracle.tau_median(confs)
    assert abs(t_gpu - t_ref) <= 2 * measure_tol(measure, rs[0]) + 1e-4


@pytest.mark.parametrize("persistent", [True, False], ids=["persistent", "per_op"])
def test_tiny_nucleus_mass(persistent):
    """The full head's probability mass ahead of the readout's token (its
    nucleus rank, Section 2), measured in the same vocabulary scan, against
    the oracle on teacher-forced fallback steps."""
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 1, TINY_P)
    toks = synth.prompts(cfg, 6, 12)
    o = oracle_for(name, 64)
    o.prefill(prompt)
    e = engine(name, 64, persistent)
    e.ee_prefill(prompt)
    inside = 0
    for i, t in enumerate(toks):
        r = o.decode_step(int(t), math.inf, 2, keep_logits=True)
        d = e.ee_decode_step_ex(math.inf, 2, int(t), -1, debug=False)
        assert not d["exited"]
        if r.gap_readout > MARGIN:
            assert d["readout_token"] == r.readout_token
            inside += check_nucleus_mass(i, d["nucleus_mass"], r.logits_full, r.readout_token) < 0.9
    print("tiny nucleus: readout token inside the 0.9 nucleus on", inside, "of", len(toks), "steps")


def _nucleus_decision_can_flip(confs, masses, cmarg, mmarg, target, t_ref):
    """Could steps within their comparison margins (a confidence within cmarg
    of a grid threshold, a mass within mmarg of 0.9) change the rule's answer
    t_ref? The answer flips if a grid threshold below t_ref could qualify or
    t_ref itself could fail: for each such threshold the acceptable fraction
    of the early answers is bounded below (uncertain steps counted against
    it) and above (uncertain steps counted for it)."""
    grid = np.arange(100, dtype=np.float32) / np.float32(100.0)
    ok_c = masses < 0.9 - mmarg
    ok_u = np.abs(masses - 0.9) <= mmarg
    for g in grid:
        if math.isfinite(t_ref) and g > np.float32(t_ref):
            break
        in_c = confs > g + cmarg
        in_u = np.abs(confs - g) <= cmarg
        e_min = in_c.sum() + (in_u & ~ok_c).sum()
        f_min = (in_c & ok_c).sum() / e_min if e_min else -1.0
        may_ok = ok_c | ok_u
        e_max = in_c.sum() + (in_u & may_ok).sum()
        f_max = ((in_c | in_u) & may_ok).sum() / e_max if e_max else -1.0
        if g == np.float32(t_ref):
            if f_min < target:
                return True
        elif f_max >= target:
            return True
    return False


@pytest.mark.parametrize("persistent", [True, False], ids=["persistent", "per_op"])
def test_tiny_nucleus_calibration(persistent):
    """The paper's calibration rule (Section 4 step four: the lowest grid
    threshold at which a fraction `target` of the early answers lie inside
    the full model's 0.9 nucleus), at the paper's 0.9 and two other targets.
    (1) The device's threshold equals the rule applied, exactly, to the
    device's own per-step record; (2) that record matches the oracle's
    confidences and nucleus masses step by step while the free-running
    sequences agree; (3) the device's threshold equals the oracle's unless a
    step within those comparison margins could change the rule's answer."""
    from paper_2609_14144_amd import EE_CAL_NUCLEUS
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompts = [synth.prompts(cfg, s, TINY_P) for s in range(100, 104)]
    confs, masses, cmarg, mmarg = [], [], [], []
    for p in prompts:
        o = oracle_for(name, 64)
        parted = False
        for r in o.generate(o.prefill(p), math.inf, 2, TINY_N, keep_logits=True):
            m = oracle.nucleus_mass_ahead(r.logits_full, r.readout_token)
            confs.append(r.conf)
            masses.append(m)
            if parted or r.gap_readout <= MARGIN:
                # past a full-head near-tie the device may decode another
                # sequence; with a readout near-tie another readout token
                cmarg.append(np.inf if parted else 1e-4 + 1e-3 * r.conf)
                mmarg.append(np.inf)
            else:
                lf = r.logits_full
                pr = np.exp(lf - lf.max())
                pr /= pr.sum()
                close = np.abs(lf - lf[r.readout_token]) <= 1e-3 * max(1.0, abs(lf[r.readout_token]))
                close[r.readout_token] = False
                cmarg.append(1e-4 + 1e-3 * r.conf)
                mmarg.append(1e-4 + 2e-3 * m + pr[close].sum())
            parted = parted or r.gap_full <= MARGIN
    confs, masses = np.array(confs, np.float32), np.array(masses)
    cmarg, mmarg = np.array(cmarg), np.array(mmarg)
    e = engine(name, 64, persistent)
    nontrivial = 0
    for target in (0.3, 0.6, 0.9):
        req = float(np.float32(target))
        t_gpu = e.ee_calibrate_threshold(prompts, TINY_N, 2, EE_CAL_NUCLEUS, target)
        dc, dm = e.ee_calibration_record(len(prompts) * TINY_N)
        # (1) the rule on the device's own record, decided in the same precision
        t_rule = oracle.tau_nucleus(dc, dm < np.float32(0.9), required=req)
        assert t_gpu == t_rule or (math.isinf(t_gpu) and math.isinf(t_rule)), (target, t_gpu, t_rule)
        nontrivial += math.isfinite(t_gpu) and t_gpu > 0.0
        # (2) the record against the oracle while the sequences agree
        known = np.isfinite(cmarg)
        assert np.all(np.abs(dc[known] - confs[known]) <= cmarg[known]), target
        sure = np.isfinite(mmarg)
        assert np.all(np.abs(dm[sure] - masses[sure]) <= mmarg[sure]), target
        # (3) the oracle's own answer
        t_ref = oracle.tau_nucleus(confs, masses < 0.9, required=req)
        flip = _nucleus_decision_can_flip(confs, masses, cmarg, mmarg, req, t_ref)
        print("nucleus target", target, "tau gpu", t_gpu, "oracle", t_ref, "can flip", flip)
        if not flip:
            assert t_gpu == t_ref or (math.isinf(t_gpu) and math.isinf(t_ref)), (target, t_gpu, t_ref)
    assert nontrivial >= 1  # at least one target pins a threshold above the bottom of the grid
    assert e.ee_position() == 0


def test_confidence_measure_rejects_unknown():
    from paper_2609_14144_amd import EEError
    e = engine("tiny_bf16", 32)
    with pytest.raises(EEError):
        e.ee_set_confidence_measure(3)


def test_tiny_free_running_matches_until_first_margin():
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    tau = tiny_tau(name)
    for seed in (1, 2, 3):
        prompt = synth.prompts(cfg, seed, TINY_P)
        o = oracle_for(name, 128)
        g0 = o.prefill(prompt)
        rs = o.generate(g0, tau, 2, TINY_N)
        e = engine(name, 128)
        assert e.ee_prefill(prompt) == g0
        tok, ex, conf = e.ee_decode_n(tau, 2, TINY_N)
        for i, r in enumerate(rs):
            gap = r.gap_readout if r.exited else r.gap_full
            if abs(r.conf - tau) <= MARGIN or gap <= MARGIN:
                break
            assert ex[i] == r.exited and tok[i] == r.token, (seed, i)
            assert abs(conf[i] - r.conf) <= 1e-4 + 1e-3 * r.conf


@pytest.mark.parametrize("name", ["tiny", "tiny_bf16"])
def test_kv_cache_contents_including_fill(name):
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 1, TINY_P)
    toks = synth.prompts(cfg, 7, 8)
    fe = np.array([1, 0, 1, 1, 0, 1, 0, 1], np.int32)
    o = oracle_for(name, 64)
    o.prefill(prompt)
    o.generate(None, 0.5, 2, 8, force_tokens=toks, force_exit=fe)
    e = engine(name, 64, page_size=16)
    e.ee_prefill(prompt)
    e.ee_decode_n_ex(0.5, 2, 8, force_tokens=toks, force_exit=fe)
    check_kv(e, o, cfg, range(cfg.n_layers), range(TINY_P + 8))


@pytest.mark.parametrize("persistent", [True, False], ids=["persistent", "per_op"])
def test_refresh_recomputes_the_cache(persistent):
    """Periodic full-depth refresh (Section 11): after a run where every token
    exits, a refresh of the decoded positions rewrites their cache entries at
    every layer as the oracle's refresh does (which equals an ungated run);
    position and next input are kept and the following steps match."""
    from paper_2609_14144_amd import EEError
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 1, TINY_P)
    toks = synth.prompts(cfg, 7, 12)
    o = oracle_for(name, 64)
    o.prefill(prompt)
    rs = o.generate(None, 0.0, 2, 12, force_tokens=toks)
    e = engine(name, 64, persistent, page_size=16)
    e.ee_prefill(prompt)
    tok, ex, conf, would = e.ee_decode_n_ex(0.0, 2, 12, force_tokens=toks)
    assert ex.all()
    o.refresh(12)
    e.ee_refresh(12)
    assert e.ee_position() == TINY_P + 12
    check_kv(e, o, cfg, range(cfg.n_layers), range(TINY_P, TINY_P + 12))
    # the next input is still the last emitted token
    nxt = o.decode_step(rs[-1].token, 0.5, 2, keep_logits=True)
    d = e.ee_decode_step_ex(0.5, 2, -1, int(nxt.exited))
    compare_step(0, d, nxt, 0.5, [])
    rep, _ = lockstep(e, o, None, 0.5, 2, 3, force_tokens=synth.prompts(cfg, 8, 3))
    for n in (0, e.ee_position() + 1):
        with pytest.raises(EEError):
            e.ee_refresh(n)


@pytest.mark.parametrize("chunk", [None, 7, 0], ids=["batched", "chunks_of_7", "stepwise"])
@pytest.mark.parametrize("name", ["tiny", "tiny_bf16"])
def test_prompt_pass_matches_oracle(name, chunk):
    """The prompt pass batched over positions (the default chunks, and chunks
    of 7 positions, whose later chunks attend to the earlier ones through
    the cache) and one position per step through the decode program: every
    layer's cache entries of every prompt position and the first token
    against the oracle's prompt pass, ragged lengths, then lockstep decode."""
    cfg = synth.get_config(name)
    for P in (1, 5, 16, 37, 200):
        prompt = synth.prompts(cfg, 60 + P, P)
        o = oracle_for(name, P + 4)
        g0 = o.prefill(prompt)
        e = engine(name, P + 4, page_size=16)
        if chunk is not None:
            e.ee_set_prefill_chunk(chunk)
        g = e.ee_prefill(prompt)
        if o.last_prefill_stats[2] > MARGIN:
            assert g == g0, (P, g, g0)
        assert e.ee_position() == P
        check_kv(e, o, cfg, range(cfg.n_layers), range(P))
        lockstep(e, o, g0, 0.5, 2, 4, force_tokens=synth.prompts(cfg, 61 + P, 4), force_exit=[1, 0, 1, 0])
        e.close()


def test_prompt_pass_is_deterministic():
    """Two batched prompt passes give identical cache bytes and tokens: the
    split-K partial sums and the attention splits are added in a fixed
    order whatever the scheduling."""
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 13, 300)
    runs = []
    for _ in range(2):
        e = engine(name, 304, page_size=16)
        g = e.ee_prefill(prompt)
        runs.append((g, _kv_all(e, cfg, range(300))))
        e.close()
    assert runs[0][0] == runs[1][0]
    np.testing.assert_array_equal(runs[0][1], runs[1][1])


@pytest.mark.timeout(900)
def test_d1p5b_refresh_matches_oracle(d15):
    """The periodic full-depth refresh at the 1.5B shape (Section 11): after
    16 imposed exits, ee_refresh(16) recomputes those positions' cache
    entries at every layer as the oracle's refresh does (16 positions: the
    matrix products split K over many workgroups at these shapes)."""
    cfg, w, prompt, o, g0 = d15
    o.reset()
    o.prefill(prompt)
    toks = synth.prompts(cfg, 21, 16)
    o.generate(None, 0.3, 14, 16, force_tokens=toks, force_exit=np.ones(16, np.int32))
    o.refresh(16)
    e = engine(D15, 512 + 64)
    e.ee_prefill(prompt)
    _, ex, _, _ = e.ee_decode_n_ex(0.3, 14, 16, force_tokens=toks, force_exit=np.ones(16, np.int32))
    assert ex.all()
    e.ee_refresh(16)
    assert e.ee_position() == 512 + 16
    check_kv(e, o, cfg, [0, 7, 14, 20, 27], range(512, 528))
    e.close()


def _kv_all(e, cfg, positions):
    out = []
    for l in range(cfg.n_layers):
        for t in positions:
            k, v = e.ee_read_kv(l, t)
            out.append(np.concatenate([k, v]))
    return np.stack(out)


@pytest.mark.parametrize("name", ["tiny_bf16", "d1p5b"])
def test_lazy_fill_is_bit_identical_to_eager(name):
    """The lazy, batched KV fill writes exactly the cache the eager fill
    writes and changes nothing else: exit bursts shorter and longer than
    one batch, a fallback after a burst, and exits still pending when the
    call returns."""
    from paper_2609_14144_amd import EE_FILL_LAZY
    cfg = synth.get_config(name)
    P = TINY_P if name == "tiny_bf16" else 64
    Le = 2 if name == "tiny_bf16" else 14
    fe = np.array([1, 1, 1, 0, 1] + [1] * 10 + [0, 0, 1, 1], np.int32)
    n = fe.size
    prompt = synth.prompts(cfg, 1, P)
    toks = synth.prompts(cfg, 7, n)
    res = {}
    for lazy in (False, True):
        e = engine(name, P + n + 4, True, page_size=16)
        if lazy:
            e.ee_set_fill_policy(EE_FILL_LAZY)
        e.ee_prefill(prompt)
        res[lazy] = (e.ee_decode_n_ex(0.5, Le, n, force_tokens=toks, force_exit=fe),
                     _kv_all(e, cfg, range(P, P + n)))
        if name == "tiny_bf16" and lazy:
            o = oracle_for(name, P + n + 4)
            o.prefill(prompt)
            o.generate(None, 0.5, Le, n, force_tokens=toks, force_exit=fe)
            check_kv(e, o, cfg, range(cfg.n_layers), range(P, P + n))
        e.close()
    for a, b in zip(res[False][0], res[True][0]):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(res[False][1], res[True][1])


def test_error_paths():
    from paper_2609_14144_amd import EEError
    name = "tiny"
    cfg = synth.get_config(name)
    e = engine(name, 24)
    with pytest.raises(EEError) as ei:
        e.ee_decode_step(0.5, 2)
    assert ei.value.code == -2  # decode before prefill
    e.ee_prefill(synth.prompts(cfg, 1, 16))
    with pytest.raises(EEError) as ei:
        e.ee_decode_step(0.5, 3)  # no readout at layer 3
    assert ei.value.code == -1
    with pytest.raises(EEError) as ei:
        e.ee_decode_step(float("nan"), 2)
    assert ei.value.code == -1
    with pytest.raises(EEError) as ei:
        e.ee_decode_step(0.5, 9)
    assert ei.value.code == -1
    with pytest.raises(EEError) as ei:
        e.ee_decode_n_ex(0.5, 2, 2, force_tokens=[0, cfg.vocab])
    assert ei.value.code == -1
    e.ee_decode_n(0.5, 2, 8)                  # fills to capacity 24
    with pytest.raises(EEError) as ei:
        e.ee_decode_step(0.5, 2)
    assert ei.value.code == -5
    with pytest.raises(EEError) as ei:
        e.ee_load_weights({"embed": np.zeros(3, np.float32)})
    assert ei.value.code == -1
    with pytest.raises(EEError) as ei:
        e.ee_load_weights({"layers.0.bogus": np.zeros(3, np.float32)})
    assert ei.value.code == -1
    e.ee_reset()
    assert e.ee_position() == 0
    assert e.ee_prefill(synth.prompts(cfg, 1, 16)) >= 0   # usable after errors
    from paper_2609_14144_amd import Engine
    e2 = Engine(cfg, 32)
    with pytest.raises(EEError) as ei:
        e2.ee_prefill([1, 2, 3])
    assert ei.value.code == -2  # weights not loaded


def test_gate_limits_and_ungated_equivalence():
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 1, TINY_P)
    toks = synth.prompts(cfg, 5, 16)
    out = {}
    for key, tau, Le in (("inf", math.inf, 2), ("ungated", 0.5, 0), ("one", 1.0, 2),
                         ("zero", 0.0, 2), ("neginf", -math.inf, 2)):
        e = engine(name, 64)
        e.ee_prefill(prompt)
        out[key] = e.ee_decode_n_ex(tau, Le, 16, force_tokens=toks)
    assert not out["inf"][1].any() and not out["one"][1].any()
    assert out["zero"][1].all() and out["neginf"][1].all()
    np.testing.assert_array_equal(out["inf"][0], out["ungated"][0])


def test_persistent_and_per_op_agree_and_are_deterministic():
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 3, TINY_P)
    tau = tiny_tau(name)
    runs = []
    for persistent in (True, True, False):
        e = engine(name, 128, persistent)
        e.ee_prefill(prompt)
        d = [e.ee_decode_step_ex(tau, 2) for _ in range(6)]
        runs.append(d)
    for a, b in zip(runs[0], runs[1]):   # run twice: identical bytes
        for k in ("token", "exited", "conf"):
            assert a[k] == b[k]
        for k in ("h_exit", "logits_readout"):
            np.testing.assert_array_equal(a[k], b[k])
    for a, b in zip(runs[0], runs[2]):   # same arithmetic per row in both programs
        assert a["token"] == b["token"] and a["exited"] == b["exited"]
        np.testing.assert_array_equal(a["h_exit"], b["h_exit"])
        np.testing.assert_array_equal(a["logits_readout"], b["logits_readout"])
        assert abs(a["conf"] - b["conf"]) <= 1e-6


def test_small_persistent_grids_cover_all_work():
    """Persistent grids of 1 and 3 workgroups: every phase loops over several
    items per workgroup (attention: 2 kv heads x 4 splits of a 1000-token
    context). Rows and tokens match the default grid and the per-op program."""
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    P = 1000
    prompt = synth.prompts(cfg, 12, P)
    tau = tiny_tau(name)
    runs = []
    for grid in (None, 1, 3, 0):
        e = engine(name, P + 8, grid != 0)
        if grid:
            e.ee_set_persistent_grid(grid)
        g = e.ee_prefill(prompt)
        d = [e.ee_decode_step_ex(tau, 2, force_exit=i % 2) for i in range(4)]
        k, v = e.ee_read_kv(cfg.n_layers - 1, P + 2)
        runs.append((g, d, k, v))
    g0, d0, k0, v0 = runs[0]
    for g, d, k, v in runs[1:]:
        assert g == g0
        np.testing.assert_array_equal(k, k0)
        np.testing.assert_array_equal(v, v0)
        for a, b in zip(d0, d):
            assert a["token"] == b["token"] and a["exited"] == b["exited"]
            np.testing.assert_array_equal(a["h_exit"], b["h_exit"])
            np.testing.assert_array_equal(a["logits_readout"], b["logits_readout"])
            assert abs(a["conf"] - b["conf"]) <= 1e-6
    o = oracle_for(name, P + 8)
    assert o.prefill(prompt) == g0 or o.last_prefill_stats[2] <= MARGIN


@pytest.mark.parametrize("page_size", [1, 16, 64])
def test_paging_ragged_prompts(page_size):
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    for P in (1, 17, 64, 65):
        prompt = synth.prompts(cfg, 40 + P, P)
        toks = synth.prompts(cfg, 41 + P, 6)
        o = oracle_for(name, P + 6)
        g0 = o.prefill(prompt)
        e = engine(name, P + 6, page_size=page_size)
        g = e.ee_prefill(prompt)
        if o.last_prefill_stats[2] > MARGIN:
            assert g == g0
        lockstep(e, o, None, 0.5, 2, 6, force_tokens=toks)


def test_calibration_matches_oracle():
    from paper_2609_14144_amd import EE_CAL_EXIT_RATE, EE_CAL_MEDIAN
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompts = [synth.prompts(cfg, s, TINY_P) for s in range(100, 108)]
    e = engine(name, 64)
    tau_med = e.ee_calibrate_threshold(prompts, TINY_N, 2, EE_CAL_MEDIAN, 0.0)
    assert abs(tau_med - tiny_tau(name)) <= 1e-4
    confs = []
    for p in prompts:
        o = oracle_for(name, 64)
        confs += [r.conf for r in o.generate(o.prefill(p), math.inf, 2, TINY_N)]
    for rate in (0.0, 0.25, 0.9, 1.0):
        t_gpu = e.ee_calibrate_threshold(prompts, TINY_N, 2, EE_CAL_EXIT_RATE, rate)
        t_ref = oracle.tau_for_exit_rate(confs, rate)
        if math.isinf(t_ref):
            assert t_gpu == t_ref
        else:
            assert abs(t_gpu - t_ref) <= 1e-4
    assert e.ee_position() == 0


@pytest.mark.parametrize("P", [4000, 8000])
def test_long_context_attention(P):
    """Long prompts at the tiny shape, ragged tails. 4000 positions: 32
    attention splits of 16 positions per wave, 8000: 32 splits of 32 positions
    per wave (the items from 4096 positions on); both more records than the
    30 that the tiny shape's merge stages in LDS at once."""
    name = "tiny_bf16"
    cfg = synth.get_config(name)
    prompt = synth.prompts(cfg, 9, P)
    o = oracle_for(name, P + 4)
    g0 = o.prefill(prompt)
    e = engine(name, P + 4, page_size=64)
    g = e.ee_prefill(prompt)
    if o.last_prefill_stats[2] > MARGIN:
        assert g == g0
    rep, _ = lockstep(e, o, g0, 0.5, 2, 4, force_exit=[0, 1, 0, 0])
    print("long-context", worst(rep))


# ---------------------------------------------------------------------------
# full-size 1.5B-shaped decoder (28 layers, H=1536, 12/2 heads, F=8960, V=151936)
# ---------------------------------------------------------------------------
D15 = "d1p5b"


@pytest.fixture(scope="module")
def d15():
    cfg = synth.get_config(D15)
    w = weights_for(D15)
    prompt = synth.prompts(cfg, 1, 512)
    o = oracle_for(D15, 512 + 64)
    g0 = o.prefill(prompt)
    return cfg, w, prompt, o, g0


def test_d1p5b_lockstep_full_size(d15):
    cfg, w, prompt, o, g0 = d15
    o.reset()
    assert o.prefill(prompt) == g0
    e = engine(D15, 512 + 64)
    assert e.ee_prefill(prompt) == g0 or o.last_prefill_stats[2] <= MARGIN
    k, v = e.ee_read_kv(27, 511)
    assert rel(k, o.kcache[27, 511].reshape(-1)) < 1e-2
    rep, outside = lockstep(e, o, g0, 0.3, 14, 8)
    print("1.5B lockstep", worst(rep), "outside-margin steps", outside)


def test_d1p5b_decode_n_imposed_exits(d15):
    """The timed entry point at full size: 16 steps in one launch with the
    oracle's tokens and imposed branches (exit rate 0.5)."""
    cfg, w, prompt, o, g0 = d15
    o.reset()
    o.prefill(prompt)
    toks = synth.prompts(cfg, 8, 16)
    fe = (np.arange(16) % 2).astype(np.int32)
    rs = o.generate(None, 0.3, 14, 16, force_tokens=toks, force_exit=fe)
    e = engine(D15, 512 + 64)
    e.ee_prefill(prompt)
    tok, ex, conf, would = e.ee_decode_n_ex(0.3, 14, 16, force_tokens=toks, force_exit=fe)
    for i, r in enumerate(rs):
        assert ex[i] == bool(fe[i])
        assert abs(conf[i] - r.conf) <= 1e-4 + 1e-3 * r.conf
        if abs(r.conf - 0.3) > MARGIN:
            assert would[i] == r.would_exit
        gap = r.gap_readout if r.exited else r.gap_full
        if gap > MARGIN:
            assert tok[i] == r.token, i


def test_d1p5b_properties():
    """Properties at full size: tau=+inf equals the ungated model token for
    token; tau<=0 exits always; both device programs give the same tokens."""
    cfg = synth.get_config(D15)
    prompt = synth.prompts(cfg, 2, 512)
    res = {}
    for key, tau, Le, pers in (("inf", math.inf, 14, True), ("ungated", 0.5, 0, True),
                               ("zero", 0.0, 14, True), ("inf_perop", math.inf, 14, False)):
        e = engine(D15, 512 + 32, pers)
        e.ee_prefill(prompt)
        res[key] = e.ee_decode_n(tau, Le, 24)
        e.close()
    np.testing.assert_array_equal(res["inf"][0], res["ungated"][0])
    np.testing.assert_array_equal(res["inf"][0], res["inf_perop"][0])
    assert not res["inf"][1].any() and res["zero"][1].all()


def test_head_kernel_planted_ties_full_vocab():
    """The fused head at V=151936: planted exact ties resolve to the lowest
    token id; argmax and max-probability match the oracle's head."""
    cfg = synth.ModelConfig("headprobe", 1, 1536, 12, 2, 128, 512, 151936, "bf16", (1,))
    w = synth.generate_weights(cfg)
    o = oracle.OracleDecoder(cfg, w, 4)
    x = np.random.default_rng(3).standard_normal(cfg.hidden).astype(np.float32)
    lg = o.full_logits(x.astype(np.float64))
    j = int(np.argmax(lg))
    for k in (0, j // 2, max(0, j - 1)):
        if k < j:
            w["embed"][k] = w["embed"][j]       # exact tie with the maximum at a lower id
            break
    o = oracle.OracleDecoder(cfg, w, 4)
    e = engine(None, 4, cfg=cfg, weights=w)
    for layer in (0, 1):
        if layer == 0:
            ref = o.full_logits(x.astype(np.float64))
        else:
            ref = o.readout_logits(x.astype(np.float64), 1)
        rj, rc, rg = oracle.head_stats(ref)
        tok, conf, logits = e.ee_head_eval(layer, x)
        assert rel(logits, ref) < 1e-4
        assert abs(conf - rc) <= 1e-5 + 1e-4 * rc
        if layer == 0:
            assert rg == 0.0 and tok == rj  # the planted tie: lowest id wins
        elif rg > MARGIN:
            assert tok == rj
        # the other two measures from the same scan (Section 10)
        m = oracle.confidence_measures(ref)
        for code, key in ((1, "margin"), (2, "negentropy")):
            e.ee_set_confidence_measure(code)
            _, c2, _ = e.ee_head_eval(layer, x, want_logits=False)
            tol = 1e-5 + 2e-4 * rc if key == "margin" else 1e-4 * (1.0 + abs(m[key]))
            assert abs(c2 - m[key]) <= tol, (layer, key, c2, m[key])
            if key == "margin" and layer == 0:
                assert c2 == 0.0  # the planted tie
        e.ee_set_confidence_measure(0)


# ---------------------------------------------------------------------------
# the other configurations at full size: 0.5B and 3B shapes, the exit-layer
# sweep of the 1.5B shape, and the long-context run with bursty exits
# ---------------------------------------------------------------------------
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["d0p5b", "d3b"])
def test_other_model_shapes_lockstep(name):
    """The 0.5B and 3B shapes (readout at half depth) after their
    configurations' 512-token prompt (five attention splits; the 0.5B shape's
    odd group of 7 query heads per KV head takes the merge path with a
    duplicated head): eight teacher-forced steps in lockstep with the oracle,
    both branches, and the exited steps' filled cache entries."""
    cfg = synth.get_config(name)
    Le = cfg.readout_layers[0]
    P = 512
    prompt = synth.prompts(cfg, 1, P)
    o = oracle_for(name, P + 8)
    g0 = o.prefill(prompt, progress=_progress(f"{name} oracle prefill of {P} positions"))
    e = engine(name, P + 8)
    g = e.ee_prefill(prompt)
    assert g == g0 or o.last_prefill_stats[2] <= MARGIN
    fe = [1, 0, 1, 1, 0, 0, 1, 0]
    rep, outside = lockstep(e, o, g0, 0.3, Le, 8, force_tokens=synth.prompts(cfg, 3, 8), force_exit=fe)
    check_kv(e, o, cfg, range(Le, cfg.n_layers, 5), [P + i for i in range(8) if fe[i]])
    print(name, worst(rep), "outside-margin steps", outside)
    e.close()


@pytest.mark.timeout(900)
def test_d1p5b_long_prompt_lockstep():
    """The 1.5B shape past 4352 positions: a 4608-token prompt, whose steps
    run the attention items of 32 positions per wave (19 splits). Eight steps
    in lockstep with the oracle with imposed branches, the prompt's cache
    entries at the last layer, and the exited steps' filled entries."""
    cfg = synth.get_config(D15)
    P = 4608
    prompt = synth.prompts(cfg, 4, P)
    o = oracle_for(D15, P + 8)
    g0 = o.prefill(prompt, progress=_progress(f"oracle prefill of {P} positions"))
    e = engine(D15, P + 8)
    g = e.ee_prefill(prompt)
    assert g == g0 or o.last_prefill_stats[2] <= MARGIN
    check_kv(e, o, cfg, [0, cfg.n_layers - 1], [0, 4351, 4352, P - 1])
    fe = [1, 0, 1, 1, 0, 0, 1, 0]
    rep, outside = lockstep(e, o, g0, 0.3, 14, 8, force_tokens=synth.prompts(cfg, 9, 8), force_exit=fe)
    check_kv(e, o, cfg, range(14, cfg.n_layers, 4), [P + i for i in range(8) if fe[i]])
    print("1.5B long prompt", worst(rep), "outside-margin steps", outside)
    e.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("Le", [7, 21])
def test_d1p5b_exit_layer_sweep(Le):
    """Readouts a quarter and three quarters deep (the exit-layer sweep of the
    1.5B shape): eight steps in one launch with imposed branches against the
    oracle, and the skipped layers' cache entries of the exited steps."""
    name = "d1p5b_sweep"
    cfg = synth.get_config(name)
    P = 256
    prompt = synth.prompts(cfg, 1, P)
    o = oracle_for(name, P + 16)
    o.prefill(prompt)
    toks = synth.prompts(cfg, 8, 8)
    fe = np.array([1, 0, 1, 1, 0, 0, 1, 0], np.int32)
    rs = o.generate(None, 0.3, Le, 8, force_tokens=toks, force_exit=fe)
    e = engine(name, P + 16)
    e.ee_prefill(prompt)
    tok, ex, conf, would = e.ee_decode_n_ex(0.3, Le, 8, force_tokens=toks, force_exit=fe)
    for i, r in enumerate(rs):
        assert ex[i] == bool(fe[i])
        assert abs(conf[i] - r.conf) <= 1e-4 + 1e-3 * r.conf
        if abs(r.conf - 0.3) > MARGIN:
            assert would[i] == r.would_exit
        gap = r.gap_readout if r.exited else r.gap_full
        if gap > MARGIN:
            assert tok[i] == r.token, i
    check_kv(e, o, cfg, range(Le, cfg.n_layers, 3), [P + i for i in range(8) if fe[i]])
    e.close()


@pytest.mark.timeout(900)
def test_d1p5b_long_context_bias_bursts():
    """Long context (8192-token prompt) with bursts of exits driven through
    the readout offset, as the long-context configuration does: a step whose
    offset is beta * e_j (e_j the unit embedding row of token j scaled by
    sqrt(H), beta = 8 sqrt(H)) exits with token j at confidence ~1; the
    two device programs agree bit for bit over the whole schedule."""
    from oracle.numerics import bf16_bits_to_f64
    cfg = synth.get_config(D15)
    w = weights_for(D15)
    P, H = 8192, cfg.hidden
    prompt = synth.prompts(cfg, 3, P)
    rng = np.random.default_rng(17)
    state, sched = 0, []
    for _ in range(24):  # two-state chain: stay 7/8 in a burst, enter one with 1/2
        state = int(rng.random() < (7 / 8 if state else 0.5))
        sched.append(state)
    targets = rng.integers(0, cfg.vocab, 24)
    tau = 0.9
    runs = {}
    for pers in (True, False):
        e = engine(D15, P + 32, pers)
        e.ee_prefill(prompt)
        out = []
        for i, (s_on, j) in enumerate(zip(sched, targets)):
            b = np.zeros(H, np.float32)
            if s_on:
                ej = bf16_bits_to_f64(w["embed"][j])
                b = (8 * math.sqrt(H) * ej / np.linalg.norm(ej) * math.sqrt(H)).astype(np.float32)
            e.ee_set_readout_bias(14, b)
            tok, exited, conf = e.ee_decode_step(tau, 14)
            if s_on:
                assert exited and tok == j and conf > 0.99, (i, tok, j, conf)
            else:
                assert exited == (conf > tau)
            out.append((tok, exited, conf))
        runs[pers] = out
        e.close()
    # tokens and branches identical; the confidence to rounding (the head's
    # vocabulary partition follows the grid, so its sums round differently)
    for a, b in zip(runs[True], runs[False]):
        assert a[:2] == b[:2] and abs(a[2] - b[2]) <= 1e-6, (a, b)
    print("long-context schedule exits", sum(x[1] for x in runs[True]), "of", len(sched))


def test_stream_probe_reads_below_the_hbm_peak():
    """The streaming-read ceiling of a buffer four times the 256 MB last-level
    cache comes from HBM: positive and below MI355X's 8 TB/s peak."""
    from paper_2609_14144_amd import EEError
    e = engine("tiny", 24)
    gbps = e.ee_stream_probe(1 << 30, 3)
    assert 1000.0 < gbps < 8000.0 * 1.02, gbps
    with pytest.raises(EEError) as ei:
        e.ee_stream_probe(8, 1)
    assert ei.value.code == -1
