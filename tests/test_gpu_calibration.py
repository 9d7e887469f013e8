"""Calibration kernels of the performance model (ws_gemm_create_calibration).

Each kind must finish without a wait timing out, and touch C only as its
contract says: the epilogue-only kernel stores a zero tile over every output
tile, the others leave C alone.  The bench-size case runs the launch the
calibration uses (8192 x 8192, full grid).
"""
from __future__ import annotations

import pytest
import torch

from tests.gpu_helpers import log

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu

SENTINEL = 12345.0


def run_kind(M, N, K, tile, stages, np_, nc, kind, load_path="registers", repeats=2):
    g = w.WsGemm(M, N, K, tile, stages, np_, nc, "bf16", load_path, calibration=kind)
    try:
        A = torch.randn(M, K, device="cuda").to(torch.bfloat16)
        B = torch.randn(K, N, device="cuda").to(torch.bfloat16)
        C = torch.full((M, N), SENTINEL, dtype=torch.float32, device="cuda")
        for _ in range(repeats):
            g(A, B, C)
        st = g.sync_status()
        return st, C
    finally:
        g.close()


CASES = [
    ((128, 128, 64), 3, 4, 4, 1024, 1024, 1024),
    ((256, 128, 64), 3, 4, 4, 1024, 1024, 2048),
    ((128, 256, 32), 4, 8, 4, 1024, 1024, 1024),
    ((64, 64, 64), 2, 8, 4, 512, 512, 512),
    ((256, 128, 64), 3, 8, 4, 768, 512, 512),
]


@pytest.mark.parametrize("load_path", ["registers", "dma"])
@pytest.mark.parametrize("kind", ["empty", "load_a", "load_b", "math", "epilogue", "load_ab"])
@pytest.mark.parametrize("tile,stages,np_,nc,M,N,K", CASES)
def test_calibration_kernel_contract(tile, stages, np_, nc, M, N, K, kind, load_path):
    log("calibration %s %s P=%d %d:%d %dx%dx%d %s" % (kind, tile, stages, np_, nc, M, N, K, load_path))
    st, C = run_kind(M, N, K, tile, stages, np_, nc, kind, load_path)
    assert st == w.WS_OK, w.ws_gemm_status_str(st)
    if kind == "epilogue":
        assert bool((C == 0).all()), "epilogue-only kernel must store a zero tile everywhere"
    else:
        assert bool((C == SENTINEL).all()), "%s kernel must not write C" % kind


@pytest.mark.parametrize("kind", ["load_a", "math", "epilogue"])
def test_calibration_at_bench_launch(kind):
    log("calibration %s at 8192^3 launch" % kind)
    st, C = run_kind(8192, 8192, 1024, (256, 128, 64), 3, 4, 4, kind, repeats=3)
    assert st == w.WS_OK
    if kind == "epilogue":
        assert bool((C == 0).all())


def test_calibration_handles_refuse_tracing():
    g = w.WsGemm(512, 512, 512, (128, 128, 64), 3, 4, 4, "bf16", calibration="math")
    try:
        buf = torch.zeros(1 << 16, dtype=torch.int32, device="cuda")
        s = w.library().ws_gemm_set_trace(g._h, w._p(buf.data_ptr()), buf.numel() * 4, 1, 4)
        assert s == w.WS_ERR_UNSUPPORTED
    finally:
        g.close()
