"""Seeded synthetic workloads (shapes, weights, KV caches) shared by the oracle and the GPU path."""
from .configs import CONFIGS, ModelShape, get  # noqa: F401
from .inputs import (  # noqa: F401
    GENERATOR_VERSION, Weights, add_w4a16, add_w8a16, bf16_bits_to_f32, f32_to_bf16_bits,
    kv_cache_shape, make_kv_cache, make_weights, pack_int4, quantize_groups4, quantize_rows, tensor_names)
