"""Scalar numerics of the oracle, in float64.

The paper does not fix a precision.  The stacks store activations and
weights in bf16 with fp32 accumulation; the oracle models that by computing in
float64 and rounding to bf16 exactly where the stored format forces it (the
normalised activation a, the SwiGLU product h and the expert output o).
"""
from __future__ import annotations

import numpy as np

BF16_MANT_BITS = 8            # significant bits, implicit leading one included
BF16_MIN_NORMAL_EXP = -126    # smallest normal exponent (same range as fp32)


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    Written from the format's definition: a normal bf16 value is m * 2^(e-7)
    with an 8-bit integer significand m, so values in [2^e, 2^(e+1)) are
    multiples of 2^(e-7); below 2^-126 the spacing stays 2^-133 (subnormals).
    Scaling by a power of two is exact in float64, and ``np.rint`` rounds
    half-way cases to even.  Overflow past the largest bf16 gives +-inf.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                      # x = f * 2^e, 0.5 <= |f| < 1
    e = e - 1                               # x in [2^e, 2^(e+1))
    e = np.maximum(e, BF16_MIN_NORMAL_EXP)  # subnormal range keeps a fixed spacing
    q = np.ldexp(1.0, (BF16_MANT_BITS - 1) - e)  # 1 / spacing
    r = np.rint(x * q) / q
    # half-way between the largest finite bf16 (255 * 2^120) and 2^128 rounds up
    # (to the even significand 256), i.e. overflows to infinity
    halfway = np.ldexp(np.float64(2 ** (BF16_MANT_BITS + 1) - 1), 127 - BF16_MANT_BITS)
    r = np.where(np.abs(x) >= halfway, np.copysign(np.inf, x), r)
    return np.where(x == 0, x, r)


def identity(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def cast_fn(dtype: str):
    """The storage cast of a stack: RNE to bf16, or none for fp32 stacks."""
    return round_bf16 if dtype == "bf16" else identity


def silu(v: np.ndarray) -> np.ndarray:
    """SiLU(v) = v * sigmoid(v) = v / (1 + exp(-v))."""
    return v / (1.0 + np.exp(-v))


def softmax_rows(z: np.ndarray) -> np.ndarray:
    """Row-wise softmax; the max shift leaves the value unchanged."""
    z = np.asarray(z, dtype=np.float64)
    ez = np.exp(z - z.max(axis=-1, keepdims=True))
    return ez / ez.sum(axis=-1, keepdims=True)
