"""bfloat16 round-to-nearest-even, from the format's definition.

bfloat16 keeps the float32 exponent range (8 exponent bits, bias 127) and 8
significant bits (7 stored + the implicit one).  A finite real x with
2^(e-1) <= |x| < 2^e is rounded to the nearest multiple of 2^(e-8); below the
smallest normal 2^-126 the spacing stays 2^-133 (subnormals).  Halfway cases go
to the even multiple.  Results above the largest finite value
(2 - 2^-7) * 2^127 become +-inf; NaN stays NaN.

Inputs are float64 (the oracle's working precision), so each value is rounded
once, directly from its float64 value.
"""
import numpy as np

BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


def round_bf16(x) -> np.ndarray:
    """Nearest bfloat16 value (ties to even), returned as float64."""
    x = np.asarray(x, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        _, e = np.frexp(x)                      # x = m * 2^e, 0.5 <= |m| < 1
        q = np.maximum(e - 8, -133)             # exponent of the rounding quantum
        r = np.ldexp(np.rint(np.ldexp(x, -q)), q)   # np.rint: half to even
        r = np.where(np.abs(r) > BF16_MAX, np.copysign(np.inf, x), r)
        r = np.where(np.isnan(x), x, r)
    return r


def bf16_bits(x) -> np.ndarray:
    """uint16 bit patterns of values that are already bfloat16 (float64 in)."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def from_bf16_bits(b) -> np.ndarray:
    """float64 values of uint16 bfloat16 bit patterns."""
    u = np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)
