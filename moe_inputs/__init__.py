"""Seeded synthetic inputs for the MoE layer workloads.

This package is shared by the tests, the benchmark and the oracle's data
scripts.  It holds the workload shapes and the recipe that draws every input
tensor from a seed; it holds none of the MoE layer's arithmetic (no routing,
no expert math).  Every tensor, and every expert slice of a per-expert tensor,
comes from its own child stream, so any slice can be regenerated on its own.
"""
from .configs import CONFIGS, config, variant, TENSOR_IDS  # noqa: F401
from .gen import (  # noqa: F401
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    gen_tensor,
    gen_expert_tensor,
    gen_expert_stack,
    layer_inputs,
    pool_size,
    stress_router_bias,
    to_f64,
)
