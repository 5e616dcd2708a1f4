"""Seeded synthetic inputs (Q/K/V tensors and logical block masks).

This package only draws inputs.  It holds none of the attention arithmetic,
so both the HIP path and the fp64 oracle can consume exactly the same bytes.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    BlockMask,
    WorkloadConfig,
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    make_mask,
    make_qkv,
    qkv_slice,
    random_case,
)
