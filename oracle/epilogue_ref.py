"""CPU oracle of the GEMM epilogue variants -- TEST INFRASTRUCTURE ONLY.

The paper's kernel stores C = A B in the accumulator type (Background,
"General Matrix Multiplication").  The library also offers the BLAS epilogue

    C <- alpha (A B) + beta C      (beta == 0: the old C is not read)

stored as binary32, bfloat16 or binary16.  This module computes that result
the plain way: the exact value in float64 (the exact product sums come from
the GEMM oracle), then one rounding to the output format, round to nearest
with ties to even, as the IEEE 754 definition of the formats states.  The
rounding is written here from the format parameters (significand precision
and exponent range), not taken from a conversion routine, so that the tests
can pin it against independent library conversions.

Only the test suite may import this module; it shares no code with the GPU
library.
"""
from __future__ import annotations

import numpy as np

# Binary floating-point formats: (precision p in bits including the leading
# one, smallest normal exponent emin, largest exponent emax).  The largest
# finite value is (2 - 2^(1-p)) 2^emax; subnormals have the fixed quantum
# 2^(emin - p + 1).
FORMATS = {
    "f32": (24, -126, 127),   # IEEE 754 binary32
    "bf16": (8, -126, 127),   # bfloat16: binary32's exponent, 8-bit significand
    "f16": (11, -14, 15),     # IEEE 754 binary16
}


def max_finite(fmt: str) -> float:
    p, _, emax = FORMATS[fmt]
    return float(np.ldexp(2.0 - np.ldexp(1.0, 1 - p), emax))


def round_to(x, fmt: str) -> np.ndarray:
    """Round float64 values to the nearest value of `fmt` (ties to even).
    Magnitudes that round beyond the largest finite value become infinities
    of the same sign; zeros, infinities and NaNs pass through.  Returns the
    rounded values as float64 (every value of the three formats is exact in
    float64)."""
    p, emin, _ = FORMATS[fmt]
    x = np.asarray(x, dtype=np.float64)
    out = x.copy()
    sel = np.isfinite(x) & (x != 0.0)
    v = x[sel]
    # v = f * 2^ex with 0.5 <= |f| < 1, so the leading bit of v has weight
    # 2^(ex - 1); below the normal range the quantum stops shrinking.
    _, ex = np.frexp(v)
    lead = np.maximum(ex - 1, emin)
    quantum = np.ldexp(1.0, lead - (p - 1))
    # v / quantum is exact (a power-of-two scaling); np.round takes halves to
    # the even integer, which is ties-to-even on the last significand bit.
    r = np.round(v / quantum) * quantum
    big = np.abs(r) > max_finite(fmt)
    r[big] = np.copysign(np.inf, v[big])
    out[sel] = r
    return out


def epilogue(AB, C_in, alpha: float, beta: float, fmt: str) -> np.ndarray:
    """alpha * AB + beta * C_in rounded once to `fmt`.  AB: the exact product
    A B (float64, from the GEMM oracle); C_in: the old C as float64 values
    (ignored when beta == 0).  alpha and beta are taken as binary32 numbers,
    as the library receives them."""
    a = float(np.float32(alpha))
    b = float(np.float32(beta))
    v = a * np.asarray(AB, dtype=np.float64)
    if b != 0.0:
        v = v + b * np.asarray(C_in, dtype=np.float64)
    return round_to(v, fmt)


def unit_roundoff(fmt: str) -> float:
    """Half a unit in the last place relative to the value: 2^-p."""
    return float(np.ldexp(1.0, -FORMATS[fmt][0]))


def epilogue_bound(absAB, C_in, alpha: float, beta: float, ref_exact, fmt: str,
                   rel: float = 1e-4) -> np.ndarray:
    """Element-wise error bound of a binary32-accumulated result rounded to
    `fmt`: the accumulation and epilogue error, at most rel * (|alpha| |A||B|
    + |beta| |C|), grown by one rounding, plus that rounding itself (2^-p of
    the exact value) and half the format's smallest subnormal."""
    p, emin, _ = FORMATS[fmt]
    u = unit_roundoff(fmt)
    scale = abs(float(np.float32(alpha))) * np.asarray(absAB, dtype=np.float64)
    if float(np.float32(beta)) != 0.0:
        scale = scale + abs(float(np.float32(beta))) * np.abs(np.asarray(C_in, dtype=np.float64))
    tiny = float(np.ldexp(1.0, emin - p))
    return rel * scale * (1.0 + u) + u * np.abs(np.asarray(ref_exact, dtype=np.float64)) + tiny
