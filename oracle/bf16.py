"""bfloat16 encode/decode for the oracle (test infrastructure only).

The attention cache stores keys and values as bfloat16 (1 sign, 8 exponent,
7 stored mantissa bits). Rotated replacement keys and queries are rounded to
that format with round-to-nearest, ties-to-even, directly from float64 (no
float32 intermediate, so there is no double rounding).
"""
import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact float64 values."""
    b = np.asarray(bits).astype(np.uint16).astype(np.uint32) << 16
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def f64_to_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bit patterns, round-to-nearest-even, from the exact value.

    A finite nonzero x is m * 2**e with 0.5 <= |m| < 1. A normal bf16 keeps 8
    significant bits, so its quantum is 2**(e - 8); below the smallest normal
    (2**-126) the quantum is fixed at 2**-133. np.rint rounds half to even, and
    x / quantum is exact because quantum is a power of two.
    """
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("oracle inputs hold no NaN/Inf")
    _, e = np.frexp(x)
    e = np.maximum(e, -125)
    quantum = np.ldexp(1.0, e - 8)
    y = np.rint(x / quantum) * quantum
    if np.any(np.abs(y) >= 2.0 ** 128):
        raise OverflowError("value outside the bf16 range")
    # y is exactly representable in bf16, hence in float32
    return (y.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
