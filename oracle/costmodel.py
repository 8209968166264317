"""Layer-equivalent cost model (Appendix C) and the estimated speedup.

One layer-equivalent is the multiply-accumulates of one decoder layer:
H*A*D + 2*H*K*D + A*D*H for the four attention projections (grouped-query
attention narrows the key and value projections) plus 3*H*F for the gated
feed-forward block. One confidence test costs H*H (readout) + H*V
(unembedding). Table C1 prints the test in layer-equivalents and as a share
of the full stack.

The estimated speedups printed in Section 5.3 (Table 3) and Section 8
(Table 4) are reproduced by S = (L + U) / (L + U - r (L - L_e)) with U = H*V
over the layer cost: the unembedding is charged on every token, the skipped
layers are credited on exits, and the confidence test run on fallback tokens
is not charged. This is a reading of the printed numbers; the prose in
Section 8 speaks of subtracting the test's cost.
"""


def layer_macs(H, A, K, D, F):
    return H * A * D + 2 * H * K * D + A * D * H + 3 * H * F


def test_macs(H, V):
    return H * H + H * V


def test_layer_equivalents(H, A, K, D, F, V):
    return test_macs(H, V) / layer_macs(H, A, K, D, F)


def test_share_of_stack(H, A, K, D, F, V, L):
    return test_layer_equivalents(H, A, K, D, F, V) / L


def estimated_speedup(H, A, K, D, F, V, L, exit_layer, exit_rate):
    U = H * V / layer_macs(H, A, K, D, F)
    return (L + U) / (L + U - exit_rate * (L - exit_layer))
