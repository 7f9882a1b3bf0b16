"""Seeded synthetic inputs shared by the CPU oracle, the GPU path, the tests and the bench.

This package only draws random tensors; it holds none of the quantization
arithmetic, so both sides of every parity check can consume the same arrays
without sharing any of the method's code.
"""

from .workloads import (CONFIGS, LLAMA3_8B, LayerConfig, config_by_name, make_layer,
                        make_triangular_problem)

__all__ = ["CONFIGS", "LLAMA3_8B", "LayerConfig", "make_layer", "make_triangular_problem",
           "config_by_name"]
