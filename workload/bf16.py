"""bfloat16 rounding from the bit layout (no ml_dtypes in this image).

bfloat16 keeps the top 16 bits of an IEEE-754 binary32 value. Rounding a
binary32 value to the nearest bfloat16, ties to even, adds 0x7FFF plus the
lowest kept bit to the 32-bit pattern and truncates. Inputs here are finite
(drawn from normal distributions), so NaN/Inf handling is not needed, but
values that would overflow are rejected loudly.
"""
import numpy as np


def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 values to bfloat16 (RNE); return the uint16 bit patterns.

    For finite inputs the 32-bit sum below cannot wrap (the largest finite
    pattern 0xFF7FFFFF plus 0x8000 stays below 2^32).
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32)
    if np.any((bits & np.uint32(0x7F800000)) == np.uint32(0x7F800000)):
        raise ValueError("bf16 rounding expects finite inputs")
    r = bits >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += bits
    r >>= np.uint32(16)
    out = r.astype(np.uint16)
    if np.any((out & np.uint16(0x7F80)) == np.uint16(0x7F80)):
        raise ValueError("value overflows bfloat16")
    return out


def bf16_bits_to_f32(bits) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to float32 exactly."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def bf16_round(a) -> np.ndarray:
    """Round to the nearest bfloat16 value and return it as float32 (exact)."""
    shape = np.shape(a)
    return bf16_bits_to_f32(f32_to_bf16_bits(np.asarray(a, dtype=np.float32).reshape(-1))).reshape(shape)
