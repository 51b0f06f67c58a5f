"""Seeded synthetic workloads for the MAP pruning hot path.

This package only draws random numbers and lays them out; it holds none of
the method's arithmetic.  Both the CPU oracle (through the tests) and the HIP
path (through the binding, tests and bench) receive the same arrays from it.
"""
from .configs import CONFIGS, PredictorShape, Workload, get_config
from .gen import (bf16_bits_to_f32, f32_to_bf16_bits, make_attention, make_inputs, make_weights,
                  make_visual_tokens, peaked_scores)

__all__ = [
    "CONFIGS", "PredictorShape", "Workload", "get_config", "make_inputs",
    "make_weights", "make_visual_tokens", "peaked_scores", "f32_to_bf16_bits",
    "bf16_bits_to_f32", "make_attention",
]
