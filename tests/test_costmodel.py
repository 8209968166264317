"""Pins of the Appendix C cost model and the estimated-speedup reading
against the values the paper prints (Tables C1, 3 and 4)."""
import os

import pytest

from oracle import costmodel

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLD, name)) as f:
        return [l.split() for l in f if l.strip() and not l.startswith("#")]


MODELS = {r[0]: tuple(int(x) for x in r[1:8]) for r in _rows("table_c1.txt")}


@pytest.mark.parametrize("row", _rows("table_c1.txt"), ids=lambda r: r[0])
def test_table_c1(row):
    H, A, K, D, F, V, L = (int(x) for x in row[1:8])
    eq = costmodel.test_layer_equivalents(H, A, K, D, F, V)
    share = 100 * costmodel.test_share_of_stack(H, A, K, D, F, V, L)
    assert f"{eq:.1f}" == row[8]
    digits = len(row[9].split(".")[1]) if "." in row[9] else 0
    assert f"{share:.{digits}f}" == row[9]


@pytest.mark.parametrize("row", _rows("speedup_tables.txt"), ids=lambda r: f"{r[0]}-{r[1]}-{r[2]}-{r[3]}")
def test_printed_speedups(row):
    """Both printed numbers are rounded (rate to 0.1 point, speedup to 0.01):
    the speedups over the rate's rounding interval must meet the speedup's."""
    H, A, K, D, F, V, L = MODELS[row[1]]
    r = float(row[3]) / 100
    lo = costmodel.estimated_speedup(H, A, K, D, F, V, L, int(row[2]), r - 0.0005)
    hi = costmodel.estimated_speedup(H, A, K, D, F, V, L, int(row[2]), r + 0.0005)
    printed = float(row[4])
    assert lo <= printed + 0.005 and hi >= printed - 0.005
    mid = costmodel.estimated_speedup(H, A, K, D, F, V, L, int(row[2]), r)
    assert abs(mid - printed) <= 0.0051


def test_layer_macs_1p5b_closed_form():
    # 2*H*A*D (q and o) + 2*H*K*D (k and v) + 3*H*F (gate, up, down)
    assert costmodel.layer_macs(1536, 12, 2, 128, 8960) == 46_792_704
