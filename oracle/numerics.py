"""bf16 storage rounding, written from the format's definition.

Oracle (test infrastructure).  bf16 has an 8-bit significand (7 stored bits
plus the implicit one) and fp32's exponent range.  Storing a real x in bf16
rounds it to the nearest multiple of the local spacing (one unit in the last
place) with ties going to the even multiple.  The KV cache is stored in bf16
for the bf16-weight models (a reading: the paper does not state precision; the
16-bit footprints it quotes in Section 5.1 are consistent with 16-bit storage).
"""
from __future__ import annotations

import numpy as np

BF16_MIN_NORMAL_EXP = -126  # smallest normal bf16 is 2**-126 (same as fp32)
BF16_SIGNIFICAND_BITS = 8


def round_bf16(x) -> np.ndarray:
    """Round each element of x (any real dtype) to the nearest bf16 value, ties to even.

    Returns float64 values that are exactly representable in bf16.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)  # x = m * 2**e with 0.5 <= |m| < 1, so x lies in [2**(e-1), 2**e)
    # spacing of bf16 values in that binade; below the normal range the spacing stays fixed
    e_eff = np.maximum(e, BF16_MIN_NORMAL_EXP + 1)
    ulp = np.ldexp(1.0, e_eff - BF16_SIGNIFICAND_BITS)
    return np.rint(x / ulp) * ulp  # np.rint rounds half to even


def bf16_bits_to_float(bits) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) to their values: the upper half of an fp32 word."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def as_float64(a) -> np.ndarray:
    """Value of a stored tensor: uint16 arrays are bf16 bit patterns, anything else is a float array."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return bf16_bits_to_float(a)
    return a.astype(np.float64)
