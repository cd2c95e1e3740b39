"""Seeded synthetic video-DiT attention inputs.

Shared by the tests, the smoke check and the benchmark: it builds Q, K, V of
the workloads' shapes and nothing else. It holds none of the routing or
attention arithmetic.
"""

from .video import (
    CONFIGS,
    WorkloadConfig,
    get_config,
    head_alphas,
    positional_embedding,
    gen_head,
    gen_qkv,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
)

__all__ = [
    "CONFIGS",
    "WorkloadConfig",
    "get_config",
    "head_alphas",
    "positional_embedding",
    "gen_head",
    "gen_qkv",
    "bf16_bits_to_f32",
    "f32_to_bf16_bits",
]
