"""Shared pieces of the GPU parity tests: run the C-ABI kernel on seeded
inputs and compare with the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from oracle.check import compare_exact, compare_tol
from paper_2506_11209_amd import inputs

REL_TOL = 1e-4  # |C - C_ref| <= 1e-4 * (|A| |B|), element-wise


def log(msg: str) -> None:
    print(msg, flush=True)


def run_gpu(A_cpu, B_cpu, tile, stages, np_, nc, dtype, C_fill=float("nan"), repeats=1,
            load_path="registers", split=0):
    """C = A B through the library on cuda:0; returns the last C as float32 numpy."""
    from paper_2506_11209_amd import wsgemm as w
    M, K = A_cpu.shape
    N = B_cpu.shape[1]
    g = w.WsGemm(M, N, K, tile, stages, np_, nc, dtype, load_path, split=split)
    try:
        A = A_cpu.cuda()
        B = B_cpu.cuda()
        C = torch.full((M, N), C_fill, dtype=torch.float32, device="cuda")
        for _ in range(repeats):
            g(A, B, C)
        st = g.sync_status()
        assert st == w.WS_OK, w.ws_gemm_status_str(st)
        return C.cpu().numpy()
    finally:
        g.close()


def check_full(C, A_cpu, B_cpu, dtype, exact):
    Cref, S = oracle.gemm(inputs.bits(A_cpu), inputs.bits(B_cpu), dtype)
    r = compare_exact(C, Cref) if exact else compare_tol(C, Cref, S, REL_TOL)
    return r


def sample_rows(M, TM, n_random=24, seed=0):
    """Rows covering the first/last row of several tile rows plus random rows."""
    rng = np.random.default_rng(seed)
    rows = {0, M - 1, TM - 1, TM, M // 2, M // 2 - 1, M - TM}
    rows |= set(rng.integers(0, M, n_random).tolist())
    return np.array(sorted(r for r in rows if 0 <= r < M), dtype=np.int64)


def check_rows(C, A_bits, B_bits, dtype, rows, ref=None, exact=False):
    if ref is None:
        ref = oracle.gemm_rows(A_bits, B_bits, dtype, rows)
    Cref, S = ref
    sub = C[rows]
    return compare_exact(sub, Cref) if exact else compare_tol(sub, Cref, S, REL_TOL)


def compare_chunked(C, ref, exact, rows_per_chunk=1024):
    """compare_exact / compare_tol over all of C, a block of rows at a time
    (bounds the temporaries for 8192 x 8192 and larger outputs)."""
    Cref, S = ref
    M = C.shape[0]
    agg = {"ok": True, "n_bad": 0, "n": 0, "max_abs_err": 0.0, "max_scaled_err": 0.0}
    for r0 in range(0, M, rows_per_chunk):
        sl = slice(r0, min(M, r0 + rows_per_chunk))
        r = compare_exact(C[sl], Cref[sl]) if exact else compare_tol(C[sl], Cref[sl], S[sl], REL_TOL)
        agg["ok"] &= r["ok"]
        agg["n_bad"] += r["n_bad"]
        agg["n"] += r["n"]
        agg["max_abs_err"] = max(agg["max_abs_err"], r["max_abs_err"])
        agg["max_scaled_err"] = max(agg["max_scaled_err"], r.get("max_scaled_err", 0.0))
    return agg
