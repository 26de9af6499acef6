"""float32 -> bfloat16 round-to-nearest-even, written from the IEEE-754 definition.

TEST INFRASTRUCTURE ONLY (the bf16 path's conversion is compared against it
bit for bit).  bfloat16 keeps the sign, the 8 exponent bits and the top 7
fraction bits of a float32.  Rounding to nearest, ties to even, on the 16
dropped bits:  add 0x7FFF plus the lowest kept bit, then truncate.  A carry out
of the fraction correctly bumps the exponent (up to infinity).  NaNs are kept
NaN by forcing a quiet fraction bit, with their sign.
"""
import numpy as np


def f32_to_bf16_bits(x) -> np.ndarray:
    u = np.ascontiguousarray(np.asarray(x, dtype=np.float32)).view(np.uint32).astype(np.uint64)
    is_nan = ((u >> 23) & 0xFF) == 0xFF
    is_nan &= (u & 0x7FFFFF) != 0
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) & 0xFFFF
    nan_bits = ((u >> 16) | 0x0040) & 0xFFFF
    return np.where(is_nan, nan_bits, r).astype(np.uint16)


def bf16_bits_to_f32(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_bf16(x) -> np.ndarray:
    """float32 values rounded to the nearest bfloat16, returned as float32."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))
