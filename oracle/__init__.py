"""CPU fp64 oracle for OJBKQ's per-layer path.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The GPU library shares no code with
this package and never imports or runs it.
"""

from . import ojbkq, philox
from .ojbkq import (NotPositiveDefinite, centres, cholesky_upper, damping, decode,
                    decode_column, dequantize, gram, jta_score, klein_alpha, klein_log_rho,
                    klein_pick, quantize_layer, reduced_residual, relaxed_solution, scales_zeros,
                    select_best)
from .philox import philox4x32_10, uniform53

__all__ = [
    "ojbkq", "philox", "NotPositiveDefinite", "centres", "cholesky_upper", "damping", "decode",
    "decode_column", "dequantize", "gram", "jta_score", "klein_alpha", "klein_log_rho", "klein_pick",
    "quantize_layer", "reduced_residual", "relaxed_solution", "scales_zeros", "select_best",
    "philox4x32_10", "uniform53",
]
