"""Pins of the epilogue oracle (oracle/epilogue_ref.py) against what the
number formats fix: independent library conversions on values they round
correctly, ties, overflow thresholds and subnormals worked out by hand from
the format definitions, and a worked epilogue example.  Each group would
catch a plausible slip in the oracle: ties away from zero, a wrong precision
or exponent range, a missing overflow, beta applied when zero."""
import numpy as np
import pytest
import torch

from oracle import epilogue_ref as E


def _fp32_samples(n=20000, seed=3):
    rng = np.random.default_rng(seed)
    # every binade that matters, signed, plus values sitting on halfway points
    mant = rng.uniform(1.0, 2.0, n)
    exps = rng.integers(-140, 128, n)
    x = np.ldexp(mant, exps) * rng.choice([-1.0, 1.0], n)
    x = x.astype(np.float32)  # inputs the library conversions see exactly
    bits = x.view(np.uint32)
    halves = (bits & ~np.uint32(0xFFFF)) | np.uint32(0x8000)  # exact bf16 ties
    return np.concatenate([x, halves.view(np.float32)])


def test_bf16_matches_torch_conversion():
    # torch's CPU float32 -> bfloat16 conversion rounds to nearest even
    x = _fp32_samples()
    x = x[np.abs(x) < 3.0e38]
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = E.round_to(x.astype(np.float64), "bf16")
    assert np.array_equal(got, want)


def test_f16_matches_numpy_conversion():
    # numpy's float64 -> float16 cast is correctly rounded (ties to even)
    rng = np.random.default_rng(5)
    x = np.ldexp(rng.uniform(1.0, 2.0, 20000), rng.integers(-30, 17, 20000))
    x *= rng.choice([-1.0, 1.0], x.size)
    with np.errstate(over="ignore"):  # values past 65520 become infinities on both sides
        want = x.astype(np.float16).astype(np.float64)
    got = E.round_to(x, "f16")
    assert np.array_equal(got, want)


def test_f32_matches_numpy_conversion():
    rng = np.random.default_rng(7)
    x = np.ldexp(rng.uniform(1.0, 2.0, 20000), rng.integers(-155, 128, 20000))
    want = x.astype(np.float32).astype(np.float64)
    assert np.array_equal(E.round_to(x, "f32"), want)


HAND_CASES = [
    # bf16: 8 significant bits, the quantum at 1 is 2^-7
    ("bf16", 1 + 2.0**-8, 1.0),                      # tie, 1.0 is even
    ("bf16", 1 + 3 * 2.0**-8, 1 + 2.0**-6),          # tie, 1 + 2^-7 is odd
    ("bf16", -(1 + 3 * 2.0**-8), -(1 + 2.0**-6)),    # ties are symmetric
    ("bf16", 1 + 2.0**-8 + 2.0**-30, 1 + 2.0**-7),   # just above the tie
    ("bf16", 255.5, 256.0),                          # 255 odd, 256 even: up
    ("bf16", 257.0, 256.0),                          # quantum 2 above 256: tie to even
    ("bf16", (2 - 2.0**-7) * 2.0**127, (2 - 2.0**-7) * 2.0**127),  # largest finite
    ("bf16", (2 - 2.0**-8) * 2.0**127, np.inf),      # halfway to 2^128: overflows
    ("bf16", 2.0**-133, 2.0**-133),                  # smallest subnormal
    ("bf16", 2.0**-134, 0.0),                        # half of it: ties to zero
    # f16: 11 significant bits, largest finite 65504, subnormal quantum 2^-24
    ("f16", 65504.0, 65504.0),
    ("f16", 65519.0, 65504.0),
    ("f16", 65520.0, np.inf),                        # halfway to 65536
    ("f16", -65520.0, -np.inf),
    ("f16", 2049.0, 2048.0),                         # quantum 2 above 2048: tie to even
    ("f16", 2051.0, 2052.0),
    ("f16", 2.0**-24, 2.0**-24),
    ("f16", 2.0**-25, 0.0),
    ("f16", 3 * 2.0**-25, 2.0**-23),                 # 1.5 quanta: tie to 2 quanta
    ("f16", 2.0**-14 - 2.0**-25, 2.0**-14),          # top of the subnormals rounds up to 2^-14
    # f32: 24 significant bits
    ("f32", 1 + 2.0**-24, 1.0),
    ("f32", 1 + 3 * 2.0**-24, 1 + 2.0**-22),
    ("f32", 2.0**-150, 0.0),
    ("f32", 3 * 2.0**-150, 2.0**-148),
]


@pytest.mark.parametrize("fmt,x,want", HAND_CASES)
def test_hand_worked_roundings(fmt, x, want):
    assert E.round_to(np.array([x]), fmt)[0] == want


def test_special_values_pass_through():
    x = np.array([0.0, -0.0, np.inf, -np.inf, np.nan])
    for fmt in E.FORMATS:
        r = E.round_to(x, fmt)
        assert r[0] == 0.0 and not np.signbit(r[0])
        assert r[1] == 0.0 and np.signbit(r[1])
        assert r[2] == np.inf and r[3] == -np.inf and np.isnan(r[4])


def test_max_finite_values():
    assert E.max_finite("f16") == 65504.0
    assert E.max_finite("bf16") == float(torch.finfo(torch.bfloat16).max)
    assert E.max_finite("f32") == float(np.finfo(np.float32).max)


def test_worked_epilogue():
    # A = [1 2], B = [3 4]^T: A B = 11; 0.5 * 11 + 2 * (-1) = 3.5
    AB = np.array([[11.0]])
    C = np.array([[-1.0]])
    for fmt in E.FORMATS:
        assert E.epilogue(AB, C, 0.5, 2.0, fmt)[0, 0] == 3.5
    # 1000.5 needs 14 significant bits: bf16 keeps 8 (quantum 4 above 512),
    # f16 11 (quantum 0.5 from 512 to 1024)
    AB = np.array([[2001.0]])
    assert E.epilogue(AB, None, 0.5, 0.0, "bf16")[0, 0] == 1000.0
    assert E.epilogue(AB, None, 0.5, 0.0, "f16")[0, 0] == 1000.5


def test_beta_zero_ignores_c():
    AB = np.array([[1.0, 2.0]])
    C = np.array([[np.nan, np.inf]])
    for fmt in E.FORMATS:
        r = E.epilogue(AB, C, 1.0, 0.0, fmt)
        assert np.array_equal(r, AB)


def test_alpha_beta_taken_as_binary32():
    # 0.1 is not a binary32 number: the library receives float(0.1f)
    a32 = float(np.float32(0.1))
    r = E.epilogue(np.array([[1.0]]), None, 0.1, 0.0, "f32")
    assert r[0, 0] == a32


def test_bound_covers_one_rounding():
    # a value exactly representable in f32 but not in bf16: the bound must
    # admit either neighbour's distance from the exact value
    ref = np.array([[1 + 2.0**-8]])
    b = E.epilogue_bound(np.array([[0.0]]), None, 1.0, 0.0, ref, "bf16")
    assert b[0, 0] >= abs(1.0 - ref[0, 0])


@pytest.mark.parametrize("mistake", ["half_away", "wrong_precision", "no_overflow", "no_subnormal"])
def test_planted_mistakes_fail_a_pin(mistake):
    """A copy of round_to with one plausible slip must disagree with at
    least one of the hand-worked cases above."""
    def bad_round(x, fmt):
        p, emin, emax = E.FORMATS[fmt]
        if mistake == "wrong_precision":
            p -= 1
        x = np.asarray(x, dtype=np.float64)
        out = x.copy()
        sel = np.isfinite(x) & (x != 0.0)
        v = x[sel]
        _, ex = np.frexp(v)
        lead = ex - 1 if mistake == "no_subnormal" else np.maximum(ex - 1, emin)
        q = np.ldexp(1.0, lead - (p - 1))
        s = v / q
        r = (np.sign(s) * np.floor(np.abs(s) + 0.5) if mistake == "half_away" else np.round(s)) * q
        if mistake != "no_overflow":
            big = np.abs(r) > np.ldexp(2.0 - np.ldexp(1.0, 1 - p), emax)
            r[big] = np.copysign(np.inf, v[big])
        out[sel] = r
        return out

    failures = sum(1 for fmt, x, want in HAND_CASES if bad_round(np.array([x]), fmt)[0] != want)
    assert failures > 0
