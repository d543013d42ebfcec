"""Seeded synthetic MTGR-shaped batches.

This package only draws inputs: jagged lengths, segment ids, timestamps and
random tensors.  It holds none of the method's arithmetic (no mask, no
attention, no normalisation), so both the CPU oracle and the HIP path can use
it without sharing any computation.
"""
from .batches import (  # noqa: F401
    CONFIGS,
    SEG_CAND,
    SEG_HIST,
    SEG_RT,
    SEG_USER,
    WINDOW,
    Layout,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_layout,
    make_values,
    round_bf16,
)
