"""Seeded synthetic inputs for the LegoLink link step.

This package is shared by the CPU oracle and by the GPU harness.  It only
draws random numbers and describes workload shapes; it contains none of the
link step's arithmetic (no token selection, no attention, no layer math).
"""
from .configs import CONFIGS, AttnWorkload, ModelWorkload, get_config  # noqa: F401
from .gen import (  # noqa: F401
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    chunk_cache,
    row_qkv,
    model_weights,
    final_norm_weight,
    token_embeddings,
    dummy_embeddings,
    matrix_bf16,
    matrix_f32,
)
