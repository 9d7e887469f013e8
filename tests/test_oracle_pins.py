"""The oracle against what the mathematics fixes (runs on the CPU)."""
import numpy as np
import pytest

import oracle
from tests import oracle_pins as pins
from paper_2506_11209_amd import inputs


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin_holds(lib, pin):
    ok, msg = pin(lib)
    assert ok, msg


def test_decode_f16_every_pattern(lib):
    b = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(b, "f16", lib=lib)
    want = pins.lib_f16_values(b)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


def test_decode_bf16_every_pattern(lib):
    b = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(b, "bf16", lib=lib)
    want = pins.lib_bf16_values(b)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])


@pytest.mark.parametrize("dtype,pattern,value", [
    ("f16", 0x3C00, 1.0), ("f16", 0xC000, -2.0), ("f16", 0x7BFF, 65504.0),
    ("f16", 0x0001, 2.0 ** -24), ("f16", 0x0400, 2.0 ** -14), ("f16", 0x3555, 0.333251953125),
    ("f16", 0x8000, -0.0), ("f16", 0x7C00, np.inf),
    ("bf16", 0x3F80, 1.0), ("bf16", 0x4049, 3.140625), ("bf16", 0x0001, 2.0 ** -133),
    ("bf16", 0x7F7F, (2 - 2.0 ** -7) * 2.0 ** 127), ("bf16", 0xFF80, -np.inf),
])
def test_decode_spot_values(lib, dtype, pattern, value):
    """Values fixed by the binary16 / bfloat16 format definitions."""
    got = oracle.decode(np.array([pattern], dtype=np.uint16), dtype, lib=lib)[0]
    assert got == value and np.signbit(got) == np.signbit(value)


def test_rows_equal_full_product(lib):
    A, B = inputs.make_operands(96, 72, 130, "bf16", "normal", 7)
    Ab, Bb = inputs.bits(A), inputs.bits(B)
    C, S = oracle.gemm(Ab, Bb, "bf16", lib=lib)
    rows = np.array([95, 0, 17, 17, 64])
    Cr, Sr = oracle.gemm_rows(Ab, Bb, "bf16", rows, lib=lib)
    assert np.array_equal(Cr, C[rows]) and np.array_equal(Sr, S[rows])


def test_threads_do_not_change_result(lib):
    A, B = inputs.make_operands(64, 48, 300, "bf16", "normal", 8)
    C1, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), "bf16", nthreads=1, lib=lib)
    C4, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), "bf16", nthreads=4, lib=lib)
    assert np.array_equal(C1, C4)


def test_degenerate_shapes(lib):
    # K = 0: the empty sum is zero
    C, S = oracle.gemm(np.zeros((3, 0), np.uint16), np.zeros((0, 5), np.uint16), "f16", lib=lib)
    assert C.shape == (3, 5) and not C.any() and not S.any()
    C, _ = oracle.gemm(np.zeros((0, 4), np.uint16), np.zeros((4, 2), np.uint16), "bf16", lib=lib)
    assert C.shape == (0, 2)


def test_bad_arguments_raise(lib):
    with pytest.raises(ValueError):
        oracle.gemm_rows(np.zeros((2, 2), np.uint16), np.zeros((2, 2), np.uint16), "f16", [2], lib=lib)
    with pytest.raises(ValueError):
        oracle.gemm(np.zeros((2, 3), np.uint16), np.zeros((2, 2), np.uint16), "f16", lib=lib)


@pytest.mark.parametrize("plant", ["ORACLE_PLANT_DROP_LAST_K", "ORACLE_PLANT_TRANSPOSE_B",
                                   "ORACLE_PLANT_SIGN"])
def test_planted_mistake_breaks_a_pin(plant):
    """A copy of the oracle with a planted mistake must fail at least one pin."""
    bad = oracle.build_variant((plant,))
    failures = [p.__name__ for p in pins.ALL_PINS if not p(bad)[0]]
    assert failures, "planted %s went unnoticed" % plant


def test_inputs_are_seeded_and_in_range():
    A1, B1 = inputs.make_operands(64, 32, 48, "f16", "int4", 1)
    A2, B2 = inputs.make_operands(64, 32, 48, "f16", "int4", 1)
    assert np.array_equal(inputs.bits(A1), inputs.bits(A2))
    assert np.array_equal(inputs.bits(B1), inputs.bits(B2))
    vals = np.unique(A1.float().numpy())
    assert set(vals.tolist()) == set(range(-4, 5))
    A3, _ = inputs.make_operands(64, 32, 48, "f16", "int4", 2)
    assert not np.array_equal(inputs.bits(A1), inputs.bits(A3))


def test_input_distributions():
    A, B = inputs.make_operands(256, 256, 1024, "bf16", "normal_k", 5)
    assert abs(float(A.float().std()) - 1 / 32) < 2e-3
    A, _ = inputs.make_operands(256, 256, 256, "bf16", "uniform", 4)
    a = A.float()
    assert float(a.min()) >= -1 and float(a.max()) <= 1 and abs(float(a.mean())) < 0.02
    A, _ = inputs.make_operands(256, 256, 256, "bf16", "normal", 3)
    assert abs(float(A.float().std()) - 1) < 0.02
