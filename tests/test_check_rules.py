"""Negative and positive controls for the acceptance rules of the parity tests
(oracle/check.py), on the CPU: every GPU parity test reduces to one of these
two functions, so each kind of mistake they must catch is planted here.

Rules (the paper's operation is the exact product C = A B, Background,
"General Matrix Multiplication"):
  * exact configurations: every fp32 output equals the fp64 oracle value;
  * floating-point configurations: |C - C_ref| <= 1e-4 (|A| |B|) element-wise,
    equality where |A| |B| is 0, and NaN / Inf fail.
"""
import numpy as np
import pytest

from oracle.check import compare_exact, compare_tol

REL = 1e-4


def _case(seed=0, shape=(48, 40)):
    rng = np.random.default_rng(seed)
    ref = rng.standard_normal(shape) * 50.0
    absab = np.abs(ref) * 3.0 + rng.uniform(1.0, 5.0, shape)
    c = ref.astype(np.float32)  # within ~6e-8 relative: accepted
    return c, ref, absab


# ---------------------------------------------------------------------------
# compare_exact
# ---------------------------------------------------------------------------
def test_exact_accepts_equal_values_and_signed_zero():
    ref = np.array([[0.0, -0.0, 3.0], [4096.0, -16.0, 2.0 ** 23]])
    c = np.array([[-0.0, 0.0, 3.0], [4096.0, -16.0, 2.0 ** 23]], dtype=np.float32)
    r = compare_exact(c, ref)
    assert r["ok"] and r["n_bad"] == 0 and r["n"] == 6


def test_exact_rejects_one_ulp_miss():
    ref = np.arange(24, dtype=np.float64).reshape(4, 6) * 7.0
    c = ref.astype(np.float32)
    c[2, 3] = np.nextafter(c[2, 3], np.float32(np.inf))
    r = compare_exact(c, ref)
    assert not r["ok"] and r["n_bad"] == 1 and r["max_abs_err"] > 0


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_exact_rejects_nan_and_inf(bad):
    ref = np.ones((3, 5))
    c = ref.astype(np.float32)
    c[1, 4] = bad
    r = compare_exact(c, ref)
    assert not r["ok"] and r["n_bad"] == 1


def test_exact_counts_every_mismatch():
    ref = np.zeros((8, 8))
    c = ref.astype(np.float32)
    c[0, 0], c[7, 7], c[3, 5] = 1.0, -1.0, np.nan
    r = compare_exact(c, ref)
    assert not r["ok"] and r["n_bad"] == 3


def test_exact_shape_mismatch_raises():
    with pytest.raises(ValueError):
        compare_exact(np.zeros((2, 3), np.float32), np.zeros((3, 2)))


# ---------------------------------------------------------------------------
# compare_tol
# ---------------------------------------------------------------------------
def test_tol_accepts_fp32_rounding_of_the_reference():
    c, ref, s = _case(1)
    r = compare_tol(c, ref, s, REL)
    assert r["ok"] and r["n_bad"] == 0 and r["max_scaled_err"] < 1e-6


def test_tol_accepts_an_error_just_inside_the_bound():
    c, ref, s = _case(2)
    c = c.astype(np.float64)
    c[5, 7] = ref[5, 7] + 0.99 * REL * s[5, 7]
    r = compare_tol(c, ref, s, REL)
    assert r["ok"] and 0.98e-4 < r["max_scaled_err"] <= REL


@pytest.mark.parametrize("factor", [2.0, 1.01])
def test_tol_rejects_an_error_beyond_the_bound(factor):
    c, ref, s = _case(3)
    c = c.astype(np.float64)
    c[10, 3] = ref[10, 3] - factor * REL * s[10, 3]
    r = compare_tol(c, ref, s, REL)
    assert not r["ok"] and r["n_bad"] == 1 and r["max_scaled_err"] > REL


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf])
def test_tol_rejects_nan_and_inf(bad):
    c, ref, s = _case(4)
    c[0, 0] = bad
    r = compare_tol(c, ref, s, REL)
    assert not r["ok"] and r["n_bad"] == 1


def test_tol_requires_equality_where_absab_is_zero():
    c, ref, s = _case(5)
    ref[2, 2], s[2, 2], c[2, 2] = 0.0, 0.0, 0.0          # zero with zero bound: fine
    ref[3, 3], s[3, 3], c[3, 3] = 0.0, 0.0, 1e-30        # any error at a zero bound: bad
    r = compare_tol(c, ref, s, REL)
    assert not r["ok"] and r["n_bad"] == 1 and r["max_scaled_err"] == np.inf


def test_tol_counts_every_mismatch_and_ignores_sign_of_error():
    c, ref, s = _case(6)
    c = c.astype(np.float64)
    for (i, j), sign in zip([(0, 1), (9, 9), (47, 39)], (1, -1, 1)):
        c[i, j] = ref[i, j] + sign * 3 * REL * s[i, j]
    r = compare_tol(c, ref, s, REL)
    assert not r["ok"] and r["n_bad"] == 3


def test_tol_detects_a_dropped_k_iteration():
    """A plausible kernel mistake: one K-iteration's contribution missing from
    one output block.  Built from a real product so the sizes are realistic."""
    rng = np.random.default_rng(7)
    A = rng.standard_normal((64, 256))
    B = rng.standard_normal((256, 64))
    ref = A @ B
    s = np.abs(A) @ np.abs(B)
    c = ref.copy()
    c[:32, :32] -= A[:32, 64:128] @ B[64:128, :32]  # drop K-iteration 1 of one 32x32 block
    r = compare_tol(c.astype(np.float32), ref, s, REL)
    assert not r["ok"] and r["n_bad"] > 900


def test_tol_shape_mismatch_raises():
    with pytest.raises(ValueError):
        compare_tol(np.zeros((2, 3)), np.zeros((2, 3)), np.zeros((3, 2)))
