"""The largest problems the planner accepts, at the edges that stress the
kernel's address arithmetic, in the benchmark's launch configuration
(256x128x64, 3 stages, 4 producer + 4 consumer waves):

  * K at the A-panel limit (256 K 2 bytes just below 2^31): 65535
    K-iterations through one tile, with a partial tile (general variant) and
    with one whole tile (plain kernel, deep-prefetch consumer); also through
    four 128x64 tiles of the two-producer-group (2:1) deep-prefetch kernel;
  * N at the C-panel limit (256 N 4 bytes just below 2^31);
  * an output of more than 2^32 bytes (M = 2^21, N = 640), with whole tiles
    (plain kernel) and with a partial last tile row (general variant).

Checked against the oracle on all rows (small M) or on sampled rows."""
import numpy as np
import pytest
import torch

import oracle
from oracle.check import compare_exact, compare_tol
from paper_2506_11209_amd import inputs
from tests.gpu_helpers import REL_TOL, log, sample_rows

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu

TILE, STAGES, NP, NC = (256, 128, 64), 3, 4, 4


def run_rows(M, N, K, dist, seed, rows, tile=TILE, stages=STAGES, np_=NP):
    A, B = inputs.make_operands(M, N, K, "bf16", dist, seed)
    g = w.WsGemm(M, N, K, tile, stages, np_, NC, "bf16")
    try:
        Ad, Bd = A.cuda(), B.cuda()
        C = torch.empty((M, N), dtype=torch.float32, device="cuda")
        g(Ad, Bd, C)
        assert g.sync_status() == w.WS_OK
        info = g.info.as_dict()
        sub = C[torch.as_tensor(rows, device="cuda")].cpu().numpy()
        del Ad, Bd, C
    finally:
        g.close()
    ref = oracle.gemm_rows(inputs.bits(A), inputs.bits(B), "bf16", rows)
    return sub, ref, info


def test_k_at_the_a_panel_limit():
    M, N, K = 3, 128, (1 << 31) // (2 * 256) - 64
    log("case max K %dx%dx%d" % (M, N, K))
    C, (Cref, S), info = run_rows(M, N, K, "normal", 41, np.arange(M))
    assert info["iters"] == K // 64 and info["general"] == 1
    r = compare_tol(C, Cref, S, REL_TOL)
    assert r["ok"], r


def test_k_at_the_a_panel_limit_whole_tiles():
    # one whole 256 x 128 tile: the plain kernel, so the deep-prefetch consumer's
    # asm K loop runs 65535 K-iterations
    M, N, K = 256, 128, (1 << 31) // (2 * 256) - 64
    log("case max K whole tile %dx%dx%d" % (M, N, K))
    rows = np.array([0, 31, 32, 127, 128, 200, 255])
    C, (Cref, S), info = run_rows(M, N, K, "normal", 44, rows)
    assert info["iters"] == K // 64 and info["general"] == 0
    r = compare_tol(C, Cref, S, REL_TOL)
    assert r["ok"], r


def test_k_at_the_a_panel_limit_two_producer_groups():
    # four whole 128 x 64 tiles of the 2:1 plain kernel (deep-prefetch consumer
    # with 168 registers a wave), 65535 K-iterations each
    M, N, K = 256, 128, (1 << 31) // (2 * 256) - 64
    log("case max K 2:1 128x64x64 %dx%dx%d" % (M, N, K))
    rows = np.array([0, 63, 127, 128, 191, 255])
    C, (Cref, S), info = run_rows(M, N, K, "normal", 45, rows, tile=(128, 64, 64), stages=4, np_=8)
    assert info["iters"] == K // 64 and info["general"] == 0 and info["split"] == 2
    r = compare_tol(C, Cref, S, REL_TOL)
    assert r["ok"], r


def test_n_at_the_c_panel_limit():
    M, N, K = 8, (1 << 31) // (4 * 256) - 128, 64
    log("case max N %dx%dx%d" % (M, N, K))
    C, (Cref, _), info = run_rows(M, N, K, "int4", 42, np.arange(M))
    assert info["tiles_n"] == N // 128
    r = compare_exact(C, Cref)
    assert r["ok"], r


@pytest.mark.parametrize("M", [1 << 21, (1 << 21) + 5], ids=["whole", "ragged"])
def test_output_beyond_4gib(M):
    N, K = 640, 64
    assert M * N * 4 > (1 << 32)
    log("case output > 4 GiB %dx%dx%d" % (M, N, K))
    rows = sample_rows(M, TILE[0], n_random=24, seed=M)
    C, (Cref, _), info = run_rows(M, N, K, "int4", 43, rows)
    assert info["general"] == (0 if M % TILE[0] == 0 else 1)
    r = compare_exact(C, Cref)
    assert r["ok"], r
