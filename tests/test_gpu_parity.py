"""Parity of the HIP kernels (through the C ABI) with the CPU oracle."""
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2506_11209_amd import inputs
from paper_2506_11209_amd.workloads import WORKLOADS, unpack
from tests.gpu_helpers import check_full, compare_chunked, log, run_gpu

pytestmark = pytest.mark.gpu

LDS_LIMIT = 163840


def fits(tile, stages):
    tm, tn, tk = tile
    return 256 + stages * 2 * (tm * tk + tk * tn) <= LDS_LIMIT


# ---------------------------------------------------------------------------
# The 256^3 fp16 small-integer workload: bit-exact.
# ---------------------------------------------------------------------------
def test_int256_f16_bit_exact():
    wl = WORKLOADS["gemm_256x256x256_f16_int4"]
    A, B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
    (tm, tn, tk, stages, np_, nc), = wl.points
    log("case int256 f16 tile=%s stages=%d np=%d nc=%d" % ((tm, tn, tk), stages, np_, nc))
    C = run_gpu(A, B, (tm, tn, tk), stages, np_, nc, wl.dtype)
    r = check_full(C, A, B, wl.dtype, exact=True)
    assert r["ok"], r


# ---------------------------------------------------------------------------
# Every compiled kernel family on small-integer operands: any indexing,
# swizzle, slot or role mistake changes an exact integer result.
# Shapes span several tiles in M and N, a ragged last round and S > stages.
# ---------------------------------------------------------------------------
FAMILIES = []
for dt in ("bf16", "f16"):
    for tk in (32, 64):
        for split in (1, 2):
            for (tm, tn) in ((32, 32), (64, 64)):
                FAMILIES.append(((tm, tn, tk), 1, split, split, dt))
            for (tm, tn) in ((64, 64), (64, 128), (128, 64), (128, 128), (128, 256), (256, 128)):
                FAMILIES.append(((tm, tn, tk), 4, 4 * split, split, dt))
                if split == 2:  # 2:1 with two groups of two producer waves
                    FAMILIES.append(((tm, tn, tk), 4, 4, 2, dt))
            # eight consumer waves, four producer waves (one group or two)
            FAMILIES.append(((256, 256, tk), 8, 4, split, dt))


@pytest.mark.parametrize("load_path", ["registers", "dma"])
@pytest.mark.parametrize("tile,nc,np_,split,dtype", FAMILIES,
                         ids=lambda x: "x".join(map(str, x)) if isinstance(x, tuple) else str(x))
def test_family_exact_on_integers(tile, nc, np_, split, dtype, load_path):
    tm, tn, tk = tile
    M, N, K = 3 * tm, 5 * tn, 7 * tk  # 15 tiles, S = 7
    stages = 2 if fits(tile, 3) is False else 3
    A, B = inputs.make_operands(M, N, K, dtype, "int4", 100 + tm + tn + tk)
    log("case family tile=%s nc=%d np=%d split=%d %s %s" % (tile, nc, np_, split, dtype, load_path))
    C = run_gpu(A, B, tile, stages, np_, nc, dtype, load_path=load_path, split=split)
    r = check_full(C, A, B, dtype, exact=True)
    assert r["ok"], r


@pytest.mark.parametrize("load_path", ["registers", "dma"])
@pytest.mark.parametrize("stages", [2, 3, 4])
@pytest.mark.parametrize("K", [64, 128, 192, 256])  # S = 1, 2, 3, 4 around the ring depth
def test_ring_depth_edges(stages, K, load_path):
    tile = (128, 128, 64)
    A, B = inputs.make_operands(256, 512, K, "bf16", "int4", 7 + K)
    log("case ring stages=%d K=%d %s" % (stages, K, load_path))
    C = run_gpu(A, B, tile, stages, 4, 4, "bf16", load_path=load_path)
    assert check_full(C, A, B, "bf16", exact=True)["ok"]


def test_single_tile_single_iteration():
    A, B = inputs.make_operands(64, 64, 32, "f16", "int4", 3)
    C = run_gpu(A, B, (64, 64, 32), 2, 1, 1, "f16")
    assert check_full(C, A, B, "f16", exact=True)["ok"]


def test_multi_round_exact():
    """512 output tiles on a 256-workgroup grid: two dispatch rounds."""
    A, B = inputs.make_operands(4096, 4096, 128, "bf16", "int4", 11)
    log("case multi-round 4096x4096x128")
    C = run_gpu(A, B, (256, 128, 64), 3, 4, 4, "bf16")
    assert check_full(C, A, B, "bf16", exact=True)["ok"]


@pytest.mark.parametrize("tile,stages,np_,nc,dtype", [
    ((256, 128, 64), 3, 4, 4, "bf16"), ((128, 256, 32), 4, 8, 4, "bf16"),
    ((128, 128, 32), 3, 4, 4, "f16"), ((64, 64, 64), 2, 2, 1, "bf16"),
])
def test_random_within_tolerance(tile, stages, np_, nc, dtype):
    A, B = inputs.make_operands(768, 1024, 1536, dtype, "normal", 21)
    log("case random tile=%s" % (tile,))
    C = run_gpu(A, B, tile, stages, np_, nc, dtype)
    r = check_full(C, A, B, dtype, exact=False)
    assert r["ok"], r


def test_output_overwritten_and_deterministic():
    A, B = inputs.make_operands(512, 512, 1024, "bf16", "normal", 5)
    C1 = run_gpu(A, B, (128, 128, 64), 3, 4, 4, "bf16", C_fill=float("nan"), repeats=1)
    C2 = run_gpu(A, B, (128, 128, 64), 3, 4, 4, "bf16", C_fill=123.0, repeats=3)
    assert np.all(np.isfinite(C1))
    assert np.array_equal(C1.view(np.uint32), C2.view(np.uint32))


# ---------------------------------------------------------------------------
# Protocol stress: injected delays force buffer-full and buffer-empty waits
# (the paper's fast / slow DMA scenarios); a tiny poll limit forces the
# watchdog, and every wave still exits.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("load_path", ["registers", "dma"])
@pytest.mark.parametrize("pdelay,cdelay", [(3, 0), (0, 3)])
def test_delays_keep_results_exact(pdelay, cdelay, load_path):
    from paper_2506_11209_amd import wsgemm as w
    A, B = inputs.make_operands(512, 512, 1024, "bf16", "int4", 9)
    log("case delays p=%d c=%d %s" % (pdelay, cdelay, load_path))
    g = w.WsGemm(512, 512, 1024, (128, 128, 64), 2, 4, 4, "bf16", load_path)
    try:
        g.set_debug(0, pdelay, cdelay)
        C = g(A.cuda(), B.cuda())
        assert g.sync_status() == w.WS_OK
        assert check_full(C.cpu().numpy(), A, B, "bf16", exact=True)["ok"]
    finally:
        g.close()


@pytest.mark.parametrize("load_path", ["registers", "dma"])
def test_watchdog_reports_timeout_then_recovers(load_path):
    from paper_2506_11209_amd import wsgemm as w
    A, B = inputs.make_operands(512, 512, 1024, "bf16", "int4", 10)
    log("case watchdog %s" % load_path)
    g = w.WsGemm(512, 512, 1024, (128, 128, 64), 2, 4, 4, "bf16", load_path)
    try:
        Ad, Bd = A.cuda(), B.cuda()
        g.set_debug(1, 20, 0)  # one poll allowed, producers ~160k cycles late
        g(Ad, Bd)
        assert g.sync_status() == w.WS_ERR_TIMEOUT
        assert g.sync_status() == w.WS_OK  # cleared
        g.set_debug(0, 0, 0)
        C = g(Ad, Bd)
        assert g.sync_status() == w.WS_OK
        assert check_full(C.cpu().numpy(), A, B, "bf16", exact=True)["ok"]
    finally:
        g.close()


def test_run_rejects_misaligned_pointers():
    from paper_2506_11209_amd import wsgemm as w
    g = w.WsGemm(256, 256, 256, (64, 64, 32), 2, 1, 1, "f16")
    try:
        buf = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
        p = buf.data_ptr()
        assert w.ws_gemm_run(g._h, p + 2, p, p, 0) == w.WS_ERR_INVALID_ARG
        assert w.ws_gemm_run(g._h, p, p + 8, p, 0) == w.WS_ERR_INVALID_ARG
        assert w.ws_gemm_run(g._h, p, p, p + 2, 0) == w.WS_ERR_INVALID_ARG
    finally:
        g.close()


# ---------------------------------------------------------------------------
# Full-size workloads, in the launch configurations the benchmark and the
# sweep time: every element of C against the oracle's full fp64 product,
# computed once per workload (the 8192^3 product takes ~20 s on 16 host
# threads) and shared by all launch points of that workload.
# ---------------------------------------------------------------------------
class _Full:
    def __init__(self, name):
        wl = WORKLOADS[name]
        self.wl = wl
        self.A, self.B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
        self.Ad, self.Bd = self.A.cuda(), self.B.cuda()
        t0 = time.time()
        self.ref = oracle.gemm(inputs.bits(self.A), inputs.bits(self.B), wl.dtype,
                               with_abs=not wl.exact)
        log("oracle %s: %.1f s on %d threads" % (name, time.time() - t0, oracle.max_threads()))


_cache = {}


def full(name):
    if name not in _cache:
        _cache.clear()
        _cache[name] = _Full(name)
    return _cache[name]


FULL_NAMES = ("gemm_4096x4096x4096_bf16_normal", "gemm_8192x8192x8192_bf16_normal",
              "gemm_8192x8192x8192_bf16_int4", "gemm_16384x256x8192_bf16_uniform",
              "gemm_2048x2048x32768_bf16_normal_k")
FULL_CASES = [(name, pt, lp) for name in FULL_NAMES
              for pt in WORKLOADS[name].points for lp in ("registers", "dma")
              if pt[4] > 0 or lp == "registers"]  # the synchronous kernel has one load path


@pytest.mark.parametrize("name,point,load_path", FULL_CASES,
                         ids=lambda x: "x".join(map(str, x)) if isinstance(x, tuple) else x)
def test_full_size_workload(name, point, load_path):
    from paper_2506_11209_amd import wsgemm as w
    tm, tn, tk, stages, np_, nc, split = unpack(point)
    f = full(name)
    wl = f.wl
    log("case full %s point=%s %s" % (name, point, load_path))
    cfg = w.config((tm, tn, tk), stages, np_, nc, wl.dtype, load_path, split)
    if not fits((tm, tn, tk), stages):
        s, _ = w.ws_gemm_create(wl.M, wl.N, wl.K, cfg)
        assert s == w.WS_ERR_LDS_OVERFLOW
        return
    g = w.WsGemm(wl.M, wl.N, wl.K, (tm, tn, tk), stages, np_, nc, wl.dtype, load_path, split=split)
    try:
        C = torch.full((wl.M, wl.N), float("nan"), dtype=torch.float32, device="cuda")
        g(f.Ad, f.Bd, C)
        g(f.Ad, f.Bd, C)
        assert g.sync_status() == w.WS_OK
        Ch = C.cpu().numpy()
        del C
    finally:
        g.close()
    r = compare_chunked(Ch, f.ref, exact=wl.exact)
    assert r["n"] == wl.M * wl.N
    assert r["ok"], r


# ---------------------------------------------------------------------------
# Event trace: results stay exact, and per K-iteration the stamps are ordered
# as the protocol requires (issue <= landed <= observed full <= release).
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("point", [(128, 128, 64, 3, 4, 4), (128, 128, 32, 4, 8, 4), (256, 256, 64, 2, 4, 8, 1),
                                   (256, 256, 32, 4, 4, 8, 2)])
def test_trace_is_ordered_and_harmless(point):
    from paper_2506_11209_amd.trace import rel, run_traced
    from paper_2506_11209_amd.workloads import Workload
    wl = Workload("trace_case", 1024, 1024, 1024, "bf16", "int4", 31, True)
    A, B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
    rec, plan, C = run_traced(wl, point, wgs=2, Ad=A.cuda(), Bd=B.cuda())
    assert check_full(C.cpu().numpy(), A, B, "bf16", exact=True)["ok"]
    n = plan["iters"] * len(range(0, plan["tiles"], plan["grid"]))
    t = rel(rec[0], n)
    ia, ib, la, lb, ready, mma, relz = (t[:, i] for i in range(7))
    assert np.all(la >= ia) and np.all(lb >= ib)
    assert np.all(ready >= np.maximum(la, lb))
    assert np.all(relz >= ready)
    assert np.all(np.diff(mma) > 0)
    if point[5] == 8:  # the generated loop's stamps: full seen, MFMAs under way, released
        assert np.all(mma >= ready) and np.all(relz >= mma)
