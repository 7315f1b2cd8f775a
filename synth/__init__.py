"""Seeded synthetic attention-layer inputs.

This module is shared by the oracle-side tests and the device-side tests and
benchmark.  It only draws and shapes random inputs (Gaussian Q/K/V, rotary
position embedding, injected attention structure, bf16 rounding); it holds none
of the sparse-attention method's own arithmetic.
"""
from .layers import (  # noqa: F401
    LayerSpec,
    SPECS,
    make_layer,
    round_to_bf16,
    bf16_bits,
    bf16_bits_to_float,
)
