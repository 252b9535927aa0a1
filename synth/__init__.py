"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle's callers.

Holds shapes, value recipes and buffer construction only; none of the
method's arithmetic lives here.
"""
from .workloads import (WORKLOADS, TINY, LLAMA3_8B, LONG_CONTEXT, SKEWED, LLAMA70B_LOOP,
                        Workload, small, SEED_BASE)
from .params import Params, default_params
from .gen import Inputs, generate, f32_to_bf16_bits, bf16_bits_to_f32

__all__ = ["WORKLOADS", "TINY", "LLAMA3_8B", "LONG_CONTEXT", "SKEWED", "LLAMA70B_LOOP",
           "Workload", "small", "SEED_BASE", "Params", "default_params", "Inputs", "generate",
           "f32_to_bf16_bits", "bf16_bits_to_f32"]
