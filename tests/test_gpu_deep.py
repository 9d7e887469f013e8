"""The generated asm K loops (ws_deep_loop.inc) in every configuration that
runs them: the deep-prefetch consumer of four consumer waves (the
generator's list: four or eight producer waves, one or two producer groups,
TK = 64 and 32) and the register-lean loop of two consumer waves per SIMD
(eight consumer waves at 256 x 256, four at 128 x 128 x 32 with two
workgroups per CU; four producer waves in one or two groups).  Their prologue, loop
bodies and last k-steps (1-8 K-iterations per tile; TK = 32 deep-consumer
tiles with an odd count take the compiler-scheduled consumer instead), slot
wrap-around at every ring depth that fits, two output tiles per workgroup,
both producer load paths, the polling path (late producers), the consumer
delay hook and the watchdog.  (The general variant keeps the
compiler-scheduled consumers.)

Operands are small integers, so every product is exact: C is compared with
the oracle on sampled rows and, over all of C, by an exact checksum
C x == A (B x) for a random +-1 vector x (fp64, integer-valued sums)."""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle.check import compare_exact
from paper_2506_11209_amd import inputs
from tests.gpu_helpers import log, sample_rows

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                                "paper_2506_11209_amd", "csrc"))
import gen_deep_loop  # noqa: E402  (the list of deep-consumer configurations)

LDS_LIMIT = 163840
# (tm, tn, tk, consumer waves, producer waves, split)
CONFIGS = ([(tm, tn, tk, nc, np_, split) for (tm, tn, tk, nc, np_) in gen_deep_loop.CONFIGS
            for split in ((1, 2) if np_ == 4 else (2,))] +
           [(tm, tn, tk, nc, np_, split) for (tm, tn, tk, nc, np_) in gen_deep_loop.ROLL_CONFIGS
            for split in (1, 2)])


def cfg_id(t):
    return "%dx%dx%d-nc%d-np%d-%d:1" % t


def max_stages(tile):
    tm, tn, tk = tile
    return (LDS_LIMIT - 256) // (2 * (tm * tk + tk * tn))


def exact_checksum(C, A, B, seed):
    rng = np.random.default_rng(seed)
    x = rng.choice([-1.0, 1.0], size=C.shape[1])
    Af = A.to(torch.float64).numpy()
    Bf = B.to(torch.float64).numpy()
    return np.array_equal(C.astype(np.float64) @ x, Af @ (Bf @ x))


def run_and_check(M, N, K, tile, stages, dtype="bf16", load_path="registers", debug=None, seed=0, split=1,
                  nc=4, np_=None):
    A, B = inputs.make_operands(M, N, K, dtype, "int4", seed)
    np_ = 4 * split if np_ is None else np_
    g = w.WsGemm(M, N, K, tile, stages, np_, nc, dtype, load_path, split=split)
    try:
        info = g.info.as_dict()
        if debug:
            g.set_debug(*debug)
        C = torch.full((M, N), float("nan"), device="cuda")
        g(A.cuda(), B.cuda(), C)
        st = g.sync_status()
        assert st == w.WS_OK, w.ws_gemm_status_str(st)
        C = C.cpu().numpy()
    finally:
        g.close()
    rows = sample_rows(M, tile[0], n_random=16, seed=seed)
    Cref, _ = oracle.gemm_rows(inputs.bits(A), inputs.bits(B), dtype, rows)
    r = compare_exact(C[rows], Cref)
    assert r["ok"], r
    assert exact_checksum(C, A, B, seed), "checksum over all of C differs"
    return info


@pytest.mark.parametrize("load_path", ["registers", "dma"])
@pytest.mark.parametrize("iters", [1, 2, 3, 4, 7, 8])
@pytest.mark.parametrize("cfg", CONFIGS, ids=cfg_id)
def test_k_iterations_and_ring_depths(cfg, iters, load_path):
    tm, tn, tk, nc, np_, split = cfg
    tile = (tm, tn, tk)
    M, N, K = 32 * tm, 32 * tn, iters * tk  # 1024 tiles: two or more per workgroup (up to 2 per CU)
    for stages in range(2, min(4, max_stages(tile)) + 1):
        log("case deep %s nc=%d np=%d %d:1 S=%d P=%d %s" % (tile, nc, np_, split, iters, stages, load_path))
        info = run_and_check(M, N, K, tile, stages, load_path=load_path, seed=100 * iters + stages,
                             split=split, nc=nc, np_=np_)
        assert info["iters"] == iters and info["general"] == 0  # the plain kernel: generated loop
        assert info["tiles"] > info["grid"], "each workgroup must take more than one tile"


@pytest.mark.parametrize("cfg", CONFIGS, ids=cfg_id)
def test_f16(cfg):
    tm, tn, tk, nc, np_, split = cfg
    log("case deep f16 %s nc=%d np=%d %d:1" % ((tm, tn, tk), nc, np_, split))
    run_and_check(8 * tm, 8 * tn, 640, (tm, tn, tk), 2, dtype="f16", seed=7, split=split, nc=nc, np_=np_)


@pytest.mark.parametrize("pdelay,cdelay", [(3, 0), (0, 3), (2, 2)])
def test_late_producers_and_consumer_delay(pdelay, cdelay):
    # late producers make the consumer's peek come up short, so it polls
    log("case deep delays p=%d c=%d" % (pdelay, cdelay))
    run_and_check(1024, 512, 768, (256, 128, 64), 3, debug=(0, pdelay, cdelay), seed=13)


@pytest.mark.parametrize("split", [1, 2])
@pytest.mark.parametrize("pdelay,cdelay", [(3, 0), (0, 3), (2, 2)])
def test_late_producers_and_consumer_delay_eight_consumers(pdelay, cdelay, split):
    log("case roll delays p=%d c=%d split=%d" % (pdelay, cdelay, split))
    run_and_check(1024, 512, 768, (256, 256, 64), 2, debug=(0, pdelay, cdelay), seed=14, split=split,
                  nc=8, np_=4)


def test_watchdog_eight_consumers():
    A, B = inputs.make_operands(1024, 512, 1024, "bf16", "int4", 18)
    log("case roll watchdog")
    g = w.WsGemm(1024, 512, 1024, (256, 256, 64), 2, 4, 8, "bf16")
    try:
        Ad, Bd = A.cuda(), B.cuda()
        g.set_debug(1, 20, 0)  # one poll allowed, producers ~160k cycles late
        g(Ad, Bd)
        assert g.sync_status() == w.WS_ERR_TIMEOUT
        assert g.sync_status() == w.WS_OK
        g.set_debug(0, 0, 0)
        C = g(Ad, Bd)
        assert g.sync_status() == w.WS_OK
        Cref, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), "bf16", with_abs=False)
        assert compare_exact(C.cpu().numpy(), Cref)["ok"]
    finally:
        g.close()


def test_watchdog_reports_timeout_then_recovers():
    A, B = inputs.make_operands(1024, 512, 1024, "bf16", "int4", 17)
    log("case deep watchdog")
    g = w.WsGemm(1024, 512, 1024, (256, 128, 64), 3, 4, 4, "bf16")
    try:
        Ad, Bd = A.cuda(), B.cuda()
        g.set_debug(1, 20, 0)  # one poll allowed, producers ~160k cycles late
        g(Ad, Bd)
        assert g.sync_status() == w.WS_ERR_TIMEOUT
        assert g.sync_status() == w.WS_OK
        g.set_debug(0, 0, 0)
        C = g(Ad, Bd)
        assert g.sync_status() == w.WS_OK
        Cref, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), "bf16", with_abs=False)
        assert compare_exact(C.cpu().numpy(), Cref)["ok"]
    finally:
        g.close()
