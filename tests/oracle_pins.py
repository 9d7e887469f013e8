"""Checks that pin the GEMM oracle to facts other than itself.

Each ``pin_*`` function takes a loaded oracle library and returns
``(ok, message)``.  ``test_oracle_pins.py`` asserts every pin holds for the
real oracle, and that each planted mistake (built into a throw-away copy of
the oracle) breaks at least one pin.
"""
from __future__ import annotations

import itertools
from fractions import Fraction

import numpy as np
import torch

import oracle


def f16_bits(x) -> np.ndarray:
    """numpy's own float -> binary16 rounding, as bit patterns."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def bf16_bits(x) -> np.ndarray:
    """torch's float32 -> bfloat16 rounding, as bit patterns."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def lib_f16_values(bits: np.ndarray) -> np.ndarray:
    """Decode binary16 with numpy (a library routine independent of the oracle)."""
    return bits.view(np.float16).astype(np.float64)


def lib_bf16_values(bits: np.ndarray) -> np.ndarray:
    """Decode bfloat16 by placing the pattern in the top half of a binary32."""
    with np.errstate(invalid="ignore"):
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def exact_product(Av, Bv):
    """Exact rational C = sum_k A[:,k] (outer) B[k,:], written as outer products."""
    M, K = Av.shape
    N = Bv.shape[1]
    C = [[Fraction(0)] * N for _ in range(M)]
    for k in range(K):
        col = [Fraction(float(Av[i, k])) for i in range(M)]
        row = [Fraction(float(Bv[k, j])) for j in range(N)]
        for i in range(M):
            if col[i] == 0:
                continue
            for j in range(N):
                C[i][j] += col[i] * row[j]
    return C


def pin_brute_force_tiny(lib, seed: int = 11):
    """Every M, N, K in {1..4}: oracle == exact rational sum of outer products."""
    rng = np.random.default_rng(seed)
    for M, N, K in itertools.product(range(1, 5), repeat=3):
        for kind in ("int_f16", "randn_bf16"):
            if kind == "int_f16":
                A = f16_bits(rng.integers(-7, 8, (M, K)))
                B = f16_bits(rng.integers(-7, 8, (K, N)))
                Av, Bv, dt = lib_f16_values(A), lib_f16_values(B), "f16"
            else:
                A = bf16_bits(rng.standard_normal((M, K)))
                B = bf16_bits(rng.standard_normal((K, N)))
                Av, Bv, dt = lib_bf16_values(A), lib_bf16_values(B), "bf16"
            C, S = oracle.gemm(A, B, dt, lib=lib)
            E = exact_product(Av, Bv)
            Eabs = exact_product(np.abs(Av), np.abs(Bv))
            for i in range(M):
                for j in range(N):
                    e, ea = E[i][j], Eabs[i][j]
                    tol = Fraction(K) * Fraction(1, 2 ** 52) * ea
                    if abs(Fraction(C[i, j]) - e) > tol or abs(Fraction(S[i, j]) - ea) > tol:
                        return False, "brute force %s M=%d N=%d K=%d at (%d,%d)" % (kind, M, N, K, i, j)
    return True, "ok"


def pin_identity(lib, seed: int = 12):
    """A I = A and I B = B, bit-exact, for random bf16 and fp16 operands."""
    rng = np.random.default_rng(seed)
    for dt, enc, dec in (("bf16", bf16_bits, lib_bf16_values), ("f16", f16_bits, lib_f16_values)):
        A = enc(rng.standard_normal((37, 29)))
        B = enc(rng.standard_normal((29, 41)))
        C, _ = oracle.gemm(A, enc(np.eye(29)), dt, lib=lib)
        if not np.array_equal(C, dec(A)):
            return False, "A I != A (%s)" % dt
        C, _ = oracle.gemm(enc(np.eye(29)), B, dt, lib=lib)
        if not np.array_equal(C, dec(B)):
            return False, "I B != B (%s)" % dt
    return True, "ok"


def pin_linearity(lib, seed: int = 13):
    """(aA1 + bA2) B == a A1 B + b A2 B and A (aB1 + bB2) == a A B1 + b A B2, exactly."""
    rng = np.random.default_rng(seed)
    M, N, K = 19, 23, 31
    A1, A2 = rng.integers(-5, 6, (M, K)), rng.integers(-5, 6, (M, K))
    B1, B2 = rng.integers(-5, 6, (K, N)), rng.integers(-5, 6, (K, N))
    a, b = 3, -2
    enc = f16_bits
    lhs, _ = oracle.gemm(enc(a * A1 + b * A2), enc(B1), "f16", lib=lib)
    r1, _ = oracle.gemm(enc(A1), enc(B1), "f16", lib=lib)
    r2, _ = oracle.gemm(enc(A2), enc(B1), "f16", lib=lib)
    if not np.array_equal(lhs, a * r1 + b * r2):
        return False, "not linear in A"
    lhs, _ = oracle.gemm(enc(A1), enc(a * B1 + b * B2), "f16", lib=lib)
    r1, _ = oracle.gemm(enc(A1), enc(B1), "f16", lib=lib)
    r2, _ = oracle.gemm(enc(A1), enc(B2), "f16", lib=lib)
    if not np.array_equal(lhs, a * r1 + b * r2):
        return False, "not linear in B"
    return True, "ok"


def pin_closed_forms(lib):
    """Closed-form sums on structured integer operands, exact."""
    for (M, N, K) in ((5, 7, 9), (16, 12, 40), (3, 64, 100)):
        i = np.arange(M)[:, None]
        j = np.arange(N)[None, :]
        kA = np.broadcast_to(np.arange(K)[None, :], (M, K))
        kB = np.broadcast_to(np.arange(K)[:, None], (K, N))
        cases = [
            (np.ones((M, K)), np.ones((K, N)), np.full((M, N), float(K))),
            (np.broadcast_to(i, (M, K)), np.broadcast_to(j, (K, N)), K * i * j * 1.0),
            (kA, np.ones((K, N)), np.full((M, N), K * (K - 1) / 2.0)),
            (kA, kB, np.full((M, N), (K - 1) * K * (2 * K - 1) / 6.0)),
        ]
        for n, (A, B, want) in enumerate(cases):
            C, _ = oracle.gemm(f16_bits(A), f16_bits(B), "f16", lib=lib)
            if not np.array_equal(C, want):
                return False, "closed form %d at %s" % (n, (M, N, K))
    return True, "ok"


def pin_transpose(lib, seed: int = 14):
    """(A B)^T == B^T A^T exactly on integer operands (also a non-square check)."""
    rng = np.random.default_rng(seed)
    for (M, N, K) in ((13, 13, 13), (8, 21, 5), (32, 32, 32)):
        A = rng.integers(-4, 5, (M, K))
        B = rng.integers(-4, 5, (K, N))
        C, _ = oracle.gemm(f16_bits(A), f16_bits(B), "f16", lib=lib)
        Ct, _ = oracle.gemm(f16_bits(B.T.copy()), f16_bits(A.T.copy()), "f16", lib=lib)
        if not np.array_equal(C.T, Ct):
            return False, "transpose at %s" % ((M, N, K),)
        # integer sums are small enough for numpy's int64 product to be exact
        if not np.array_equal(C, (A @ B).astype(np.float64)):
            return False, "integer product at %s" % ((M, N, K),)
    return True, "ok"


def pin_abs_sum(lib, seed: int = 15):
    """|A| |B| equals the product of the sign-cleared operands and bounds |A B|."""
    rng = np.random.default_rng(seed)
    A = bf16_bits(rng.standard_normal((24, 40)))
    B = bf16_bits(rng.standard_normal((40, 33)))
    C, S = oracle.gemm(A, B, "bf16", lib=lib)
    Cabs, _ = oracle.gemm(A & 0x7FFF, B & 0x7FFF, "bf16", lib=lib)
    if not np.array_equal(S, Cabs):
        return False, "absAB != |A||B|"
    if np.any(np.abs(C) > S):
        return False, "|C| > absAB"
    return True, "ok"


def pin_library_dgemm(lib, seed: int = 16):
    """Against numpy's float64 matmul on decoded operands (a BLAS dgemm)."""
    rng = np.random.default_rng(seed)
    A = bf16_bits(rng.standard_normal((64, 96)))
    B = bf16_bits(rng.standard_normal((96, 80)))
    C, S = oracle.gemm(A, B, "bf16", lib=lib)
    ref = lib_bf16_values(A) @ lib_bf16_values(B)
    if np.any(np.abs(C - ref) > 1e-13 * S):
        return False, "differs from numpy dgemm"
    return True, "ok"


ALL_PINS = (pin_brute_force_tiny, pin_identity, pin_linearity, pin_closed_forms, pin_transpose,
            pin_abs_sum, pin_library_dgemm)
