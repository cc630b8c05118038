"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package holds no arithmetic of the PIPO method itself: it only defines the
model shapes of the benchmark workloads, a counter-based random generator
(SplitMix64) and the recipes that turn it into weights, prompts and the uniform
draws a sampler consumes.  The HIP library implements the same generator on
the device from the same published definition; the two implementations share
no code.
"""
from .rspec import (  # noqa: F401
    splitmix64, key, weight_values, weight_tensor, bf16_round, bf16_bits,
    prompt_tokens, uniform_draw, gain_values, TENSOR_IDS, layer_tid,
)
from .configs import ModelConfig, Workload, WORKLOADS, model_tensor_shapes  # noqa: F401
