"""Seeded synthetic inputs shared by the CPU oracle, the GPU path, the tests and the bench.

This package only draws random tensors; it holds none of the quantization
arithmetic, so both sides of every parity check can consume the same arrays
without sharing any of the method's code.
"""

from .workloads import CONFIGS, LayerConfig, make_layer, make_triangular_problem, config_by_name

__all__ = ["CONFIGS", "LayerConfig", "make_layer", "make_triangular_problem", "config_by_name"]
