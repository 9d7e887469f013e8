"""Comparison of a GPU result with the oracle -- TEST INFRASTRUCTURE ONLY.

Acceptance rules for the GEMM (all in float64):
* exact configs (small-integer operands): every fp32 output equals the fp64
  oracle value, which is an integer below 2^24 and hence exactly representable;
* floating-point configs: |C - C_ref| <= rel * (|A| |B|) element-wise with
  rel = 1e-4; where |A| |B| is zero, equality is required.  NaN / Inf fail.
"""
from __future__ import annotations

import numpy as np


def compare_exact(C, C_ref) -> dict:
    c = np.asarray(C, dtype=np.float64)
    r = np.asarray(C_ref, dtype=np.float64)
    if c.shape != r.shape:
        raise ValueError("shape mismatch %s vs %s" % (c.shape, r.shape))
    bad = ~(c == r)
    # equal infinities are no error; the largest error is over the mismatches
    with np.errstate(invalid="ignore"):
        err = float(np.max(np.abs(c[bad] - r[bad]))) if bad.any() else 0.0
    return {"ok": not bool(bad.any()), "n_bad": int(bad.sum()), "n": int(c.size), "max_abs_err": err}


def compare_tol(C, C_ref, absAB, rel: float = 1e-4) -> dict:
    c = np.asarray(C, dtype=np.float64)
    r = np.asarray(C_ref, dtype=np.float64)
    s = np.asarray(absAB, dtype=np.float64)
    if c.shape != r.shape or c.shape != s.shape:
        raise ValueError("shape mismatch %s / %s / %s" % (c.shape, r.shape, s.shape))
    err = np.abs(c - r)
    finite = np.isfinite(c)
    bound = rel * s
    bad = ~finite | (err > bound)
    with np.errstate(divide="ignore", invalid="ignore"):
        scaled = np.where(s > 0, err / np.where(s > 0, s, 1.0), np.where(err > 0, np.inf, 0.0))
    return {"ok": not bool(bad.any()), "n_bad": int(bad.sum()), "n": int(c.size),
            "max_scaled_err": float(np.max(scaled)) if c.size else 0.0,
            "max_abs_err": float(np.max(err)) if c.size else 0.0}
