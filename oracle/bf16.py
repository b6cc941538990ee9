"""bfloat16 <-> float64 conversions for the oracle (test infrastructure only).

bfloat16 is the upper half of an IEEE binary32: decoding widens the 16 stored
bits to a binary32 and then to binary64, which is exact.
"""

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (uint16/int16 array) as float64."""
    u = np.asarray(bits).astype(np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (nearest, ties to even) via exact steps.

    Used only by the oracle's tests to state what a correctly rounded bfloat16
    result is; the rounding is done on the float64 value directly (no double
    rounding through float32): the bfloat16 grid spacing at the value's binade
    is computed and ``numpy.rint`` (ties to even) is applied in that unit.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros(x.shape, np.float64)
    nz = (x != 0) & np.isfinite(x)
    e = np.floor(np.log2(np.abs(x[nz])))
    # guard against log2 rounding at exact powers of two
    e = np.where(np.abs(x[nz]) < 2.0 ** e, e - 1, e)
    e = np.where(np.abs(x[nz]) >= 2.0 ** (e + 1), e + 1, e)
    e = np.maximum(e, -126)  # subnormal range keeps the same spacing
    ulp = 2.0 ** (e - 7)
    out[nz] = np.rint(x[nz] / ulp) * ulp
    out[~np.isfinite(x)] = x[~np.isfinite(x)]
    f32 = out.astype(np.float32)  # exact: out is representable in bfloat16
    return (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
