"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and the bench.

This package holds no arithmetic of the decode method itself: it only draws random
keys, values and queries, rounds them to the storage dtype, and lays them out.
"""
from .synth import (  # noqa: F401
    CONFIGS,
    Config,
    LayerInputs,
    bf16_bits_to_f32,
    bits_to_f64,
    f32_to_bf16_bits,
    f32_to_dtype_bits,
    hot_pages,
    layer_inputs,
    page_table_permutation,
    query_trajectory,
    prefill_trajectory,
    to_physical,
)
