"""Threshold calibration (Section 4, step four).

The paper calibrates offline on a held-out sample of deployment traffic run
through the unmodified model: for every token it records the readout's
confidence and whether the readout's choice lies inside the full model's 0.9
nucleus, then takes the lowest threshold at which 90 percent of the early
answers are acceptable. The synthetic models have no traffic whose fidelity
means anything, so runs are also calibrated to a target exit rate.

Readings:
  * Exit-rate mode: sort the n recorded confidences ascending c_(1)..c_(n),
    k = floor(r*n + 1/2); tau = c_(n-k) for 0 < k < n, +inf for k = 0, -inf for
    k = n. Replaying the same tokens then exits exactly k times (c > tau) when
    no confidences tie.
  * Median mode: tau = numpy median of the confidences, as fp32.
  * Nucleus (Section 2 "Nucleus", "Acceptance"): order tokens by probability
    descending, then id ascending; the nucleus is the shortest prefix of that
    order whose mass reaches 0.9, so token j is inside iff the mass strictly
    ahead of j is below 0.9. Threshold grid 0.00, 0.01, ..., 0.99 (the paper
    prints two-decimal thresholds); the smallest grid value whose early answers
    (c > tau) are at least 90 percent acceptable; an empty early set does not
    qualify; +inf when no grid value qualifies.
All thresholds are returned as fp32 values, matching the gate's comparison.
"""
import math

import numpy as np


def tau_for_exit_rate(confs, rate: float) -> float:
    c = np.sort(np.asarray(confs, dtype=np.float32))
    n = c.size
    if n == 0:
        raise ValueError("no confidences")
    if not (0.0 <= rate <= 1.0):
        raise ValueError("rate outside [0, 1]")
    k = int(math.floor(rate * n + 0.5))
    if k == 0:
        return math.inf
    if k == n:
        return -math.inf
    return float(c[n - k - 1])


def tau_median(confs) -> float:
    return float(np.float32(np.median(np.asarray(confs, dtype=np.float32).astype(np.float64))))


def nucleus_mass_ahead(logits_full: np.ndarray, token: int) -> float:
    """Full-model probability mass strictly ahead of token in the order
    (probability descending, id ascending)."""
    z = logits_full - logits_full.max()
    p = np.exp(z)
    p /= p.sum()
    pj = p[token]
    return float(p[(p > pj) | ((p == pj) & (np.arange(p.size) < token))].sum())


def nucleus_acceptable(logits_full: np.ndarray, token: int, top_p: float = 0.9) -> bool:
    return nucleus_mass_ahead(logits_full, token) < top_p


def tau_nucleus(confs, acceptable, required: float = 0.9) -> float:
    c = np.asarray(confs, dtype=np.float32)
    ok = np.asarray(acceptable, dtype=bool)
    for i in range(100):
        tau = np.float32(i / 100.0)
        early = c > tau
        if early.any() and ok[early].mean() >= required:
            return float(tau)
    return math.inf
