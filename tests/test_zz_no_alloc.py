"""The allocation-free decode entry point (ee_decode_n_noalloc) against
ee_decode_n through the C ABI: identical tokens, exit decisions and
confidences on two calls in a row (the second shorter), a sequence that
continues identically afterwards, and the error for a working set larger
than the library-resident scratch."""
import math

import numpy as np
import pytest

import synth
from tests.gpu_helpers import engine

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _outputs(n):
    import torch
    return (torch.full((n,), -7, dtype=torch.int32, device="cuda"),
            torch.full((n,), -7, dtype=torch.int32, device="cuda"),
            torch.full((n,), float("nan"), dtype=torch.float32, device="cuda"))


@pytest.mark.parametrize("name,persistent", [("tiny_bf16", True), ("tiny_bf16", False), ("d1p5b", True)],
                         ids=["tiny_persistent", "tiny_per_op", "d1p5b_persistent"])
def test_noalloc_matches_decode_n(name, persistent):
    import torch
    cfg = synth.get_config(name)
    P = 16 if name.startswith("tiny") else 512
    Le = cfg.readout_layers[0]
    prompt = synth.prompts(cfg, 1, P)
    a = engine(name, P + 64, persistent)
    b = engine(name, P + 64, persistent)
    # tau: the median readout confidence of a full-depth run, so both branches occur
    a.ee_prefill(prompt)
    tau = float(np.median(a.ee_decode_n(math.inf, Le, 16)[2]))
    a.ee_reset()
    assert a.ee_prefill(prompt) == b.ee_prefill(prompt)
    exits = steps = 0
    for n in (24, 7):
        tok, ex, conf = a.ee_decode_n(tau, Le, n)
        dt, de, dc = _outputs(n)
        b.ee_decode_n_noalloc(tau, Le, n, dt.data_ptr(), de.data_ptr(), dc.data_ptr())
        torch.cuda.synchronize()
        np.testing.assert_array_equal(dt.cpu().numpy(), tok)
        np.testing.assert_array_equal(de.cpu().numpy(), ex.astype(np.int32))
        np.testing.assert_array_equal(dc.cpu().numpy(), conf)
        assert a.ee_position() == b.ee_position() == P + steps + n
        exits += int(ex.sum())
        steps += n
    assert 0 < exits < steps
    # the sequence state (cache, next input) continues as after ee_decode_n
    ra, rb = a.ee_decode_n(tau, Le, 5), b.ee_decode_n(tau, Le, 5)
    for x, y in zip(ra, rb):
        np.testing.assert_array_equal(x, y)
    a.close()
    b.close()


def test_noalloc_rejects_a_working_set_beyond_the_scratch():
    """A context whose attention partial records alone exceed the 4 MiB
    scratch (tiny shape, 262144 positions: 2048 splits of 2 x 132 words)
    gets EE_ECAPACITY; the context stays usable through ee_decode_n."""
    from paper_2609_14144_amd import EEError
    cfg = synth.get_config("tiny_bf16")
    e = engine("tiny_bf16", 262144)
    e.ee_prefill(synth.prompts(cfg, 1, 16))
    dt, de, dc = _outputs(4)
    with pytest.raises(EEError) as ei:
        e.ee_decode_n_noalloc(0.5, 2, 4, dt.data_ptr(), de.data_ptr(), dc.data_ptr())
    assert ei.value.code == -5 and "scratch" in str(ei.value)
    assert e.ee_position() == 16
    tok, ex, conf = e.ee_decode_n(0.5, 2, 4)
    assert e.ee_position() == 20 and np.all(np.isfinite(conf))
    with pytest.raises(EEError) as ei:
        e.ee_decode_n_noalloc(0.5, 2, 4, 0, de.data_ptr(), dc.data_ptr())
    assert ei.value.code == -1
    e.close()
