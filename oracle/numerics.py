"""bf16 and fp8 (E4M3) storage rounding, written from the formats' definitions.

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


# OCP FP8 E4M3 ("fn": no infinities): 1 sign bit, 4 exponent bits with bias 7, 3 fraction
# bits.  Normal values (1 + f/8) 2^(e-7) for e = 1..15 except the NaN code e = 15, f = 7, so
# the largest finite value is 1.75 * 2^8 = 448; subnormals f/8 * 2^-6 for e = 0.
E4M3_MAX = 448.0
E4M3_MIN_NORMAL_EXP = -6
E4M3_SIGNIFICAND_BITS = 4


def round_fp8_e4m3(x) -> np.ndarray:
    """Round each element of x to the nearest E4M3 value, ties to even; magnitudes that round
    beyond 448 saturate to 448 (the saturating conversion); NaN stays NaN.

    Returns float64 values that are exactly representable in E4M3.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    e_eff = np.maximum(e, E4M3_MIN_NORMAL_EXP + 1)
    ulp = np.ldexp(1.0, e_eff - E4M3_SIGNIFICAND_BITS)
    r = np.rint(x / ulp) * ulp
    return np.clip(r, -E4M3_MAX, E4M3_MAX)


def fp8_e4m3_bits_to_float(bits) -> np.ndarray:
    """Decode E4M3 bit patterns (uint8) to their values."""
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    s = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 15
    f = b & 7
    mag = np.where(e == 0, np.ldexp(f.astype(np.float64), -9), np.ldexp(1.0 + f / 8.0, e - 7))
    mag = np.where((e == 15) & (f == 7), np.nan, mag)
    return s * mag


def bf16_bits_to_float(bits) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) to their values: the upper half of an fp32 word."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def as_float64(a) -> np.ndarray:
    """Value of a stored tensor: uint16 arrays are bf16 bit patterns, uint8 arrays E4M3 bit
    patterns, anything else is a float array."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return bf16_bits_to_float(a)
    if a.dtype == np.uint8:
        return fp8_e4m3_bits_to_float(a)
    return a.astype(np.float64)


def as_dtype(a, dtype) -> np.ndarray:
    """Value of a stored tensor (as as_float64) in the given float type.  bf16 bit patterns go
    to float32 exactly (a bf16 value is the upper half of an fp32 word), then to `dtype`."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(dtype, copy=False)
    return as_float64(a).astype(dtype, copy=False)
