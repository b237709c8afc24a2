"""bfloat16 storage conversions (data format only).

bf16 is the upper half of an IEEE float32.  Rounding float32 to bf16 uses
round-to-nearest-even on the 16 discarded bits.  NaN is not produced by any
generator here, so it gets no special case.
"""
import numpy as np


def f32_to_bf16_bits(x):
    """float32 array -> uint16 bf16 bit patterns, round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b):
    """uint16 bf16 bit patterns -> float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)
