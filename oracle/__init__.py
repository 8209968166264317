"""CPU oracle for the batch-1 early-exit decode step.

TEST INFRASTRUCTURE ONLY. Only the test suite, the package's smoke check and
the benchmark's CPU-baseline leg may import, call or execute anything here.
The product path (the HIP library and its Python binding) never touches it.

Plain, slow, fp64 numpy written from the paper's definitions:
  * decoder layer: four attention projections with grouped-query attention and
    three gated feed-forward matrices (Appendix C cost model);
  * readout: a square matrix plus an offset applied to the exit-layer residual
    stream, whose result goes through the model's own final normalisation and
    unembedding unchanged (Section 2 "Readout, or lens"; Section 4 step two;
    Appendix B);
  * confidence gate: emit the readout's best token when its softmax
    probability exceeds the threshold, otherwise run the remaining layers
    (Section 2 "Confidence gate"; Section 4 step five);
  * KV-absence fill: the skipped layers' cache entries are the exit-layer state
    projected through those layers' key and value matrices (Section 4 step
    five);
  * threshold calibration (Section 4 step four) and the layer-equivalent cost
    model (Appendix C).
Readings where the paper is silent are listed in the module docstrings.

Parity status: every function is pinned by tests under tests/ (test_oracle_*).
"""
from .numerics import round_to_storage, rmsnorm, rope, silu, head_stats, confidence_measures, MEASURES
from .decoder import OracleDecoder, StepResult
from .calibrate import tau_for_exit_rate, tau_median, nucleus_acceptable, nucleus_mass_ahead, tau_nucleus
from . import costmodel

__all__ = ["OracleDecoder", "StepResult", "round_to_storage", "rmsnorm", "rope", "silu",
           "head_stats", "tau_for_exit_rate", "tau_median", "nucleus_acceptable",
           "tau_nucleus", "costmodel"]
