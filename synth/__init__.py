"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

This package holds no part of the decoding method's arithmetic. It only
defines model shapes, workload recipes and one counter-based random number
generator with two bit-identical backends (numpy on the host, torch on any
device), so that both sides of every parity test start from the same bytes.
"""
from .inputs import (  # noqa: F401
    ModelShape, TINY, B8, fnv1a64, counter_u64_np, counter_u64_torch,
    weight_np, weight_torch, tokens_np, tokens_torch, uniform01_np,
    hidden_np, bf16_bits_to_f32, f32_to_bf16_bits, WEIGHT_NAMES,
    model_weights_np, model_weights_torch, position_scales_np,
)
from .workloads import WORKLOADS, Workload  # noqa: F401
