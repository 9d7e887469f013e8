"""Empty problems (M, N or K = 0) through the C-ABI: nothing launches for
M or N = 0, and K = 0 writes the epilogue of the empty sum, C <- beta C
(zeros by default), checked against the oracle (its product over K = 0 is
the empty sum) and oracle/epilogue_ref.py."""
import numpy as np
import pytest
import torch

import oracle
from oracle import epilogue_ref as E
from oracle.check import compare_exact
from paper_2506_11209_amd import inputs
from tests.gpu_helpers import log

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu

GUARD = 1024
SENTINEL = -7.0
TORCH_OUT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
CONFIGS = [((256, 128, 64), 3, 4, 4), ((64, 64, 32), 3, 2, 1), ((128, 128, 32), 2, 0, 4)]


def handle(M, N, K, config, dtype="bf16"):
    tile, stages, np_, nc = config
    g = w.WsGemm(M, N, K, tile, stages, np_, nc, dtype)
    assert g.info.grid == 0
    return g


@pytest.mark.parametrize("config", CONFIGS, ids=lambda c: "%s-%d-%d" % ("x".join(map(str, c[0])), c[2], c[3]))
@pytest.mark.parametrize("M,N,K", [(0, 64, 64), (64, 0, 64), (0, 0, 0), (0, 8, 0)])
def test_no_output_means_nothing_to_do(M, N, K, config):
    log("case empty %dx%dx%d %s" % (M, N, K, config))
    g = handle(M, N, K, config)
    try:
        guard = torch.full((GUARD,), SENTINEL, device="cuda")
        # pointers to empty matrices may be NULL; a real buffer must stay untouched
        for c_ptr in (0, guard.data_ptr()):
            assert w.ws_gemm_run(g._h, 0, 0, c_ptr, 0) == w.WS_OK
        assert g.sync_status() == w.WS_OK
        assert bool((guard == SENTINEL).all())
    finally:
        g.close()


@pytest.mark.parametrize("config", CONFIGS, ids=lambda c: "%s-%d-%d" % ("x".join(map(str, c[0])), c[2], c[3]))
@pytest.mark.parametrize("M,N", [(1, 8), (300, 136), (2048, 1000)])
def test_k_zero_writes_zeros(M, N, config):
    log("case empty K=0 %dx%d %s" % (M, N, config))
    g = handle(M, N, 0, config)
    try:
        buf = torch.full((M * N + GUARD,), float("nan"), device="cuda")
        buf[M * N:] = SENTINEL
        assert w.ws_gemm_run(g._h, 0, 0, buf.data_ptr(), 0) == w.WS_OK
        assert g.sync_status() == w.WS_OK
        out = buf.cpu().numpy()
        ref, _ = oracle.gemm(np.zeros((M, 0), np.uint16), np.zeros((0, N), np.uint16), "bf16")
        assert compare_exact(out[:M * N].reshape(M, N), ref)["ok"]
        assert np.all(out[M * N:] == SENTINEL)
    finally:
        g.close()


@pytest.mark.parametrize("out", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("alpha,beta", [(1.0, 0.0), (3.0, -2.0), (0.5, 0.25)])
def test_k_zero_epilogue(alpha, beta, out):
    M, N = 129, 264
    log("case empty K=0 epilogue alpha=%g beta=%g out=%s" % (alpha, beta, out))
    g = handle(M, N, 0, CONFIGS[0])
    try:
        g.set_epilogue(alpha, beta, out)
        C_in = inputs.make_output(M, N, out, "int4", 17)
        buf = torch.full((M * N + GUARD,), SENTINEL, dtype=TORCH_OUT[out])
        buf[:M * N] = C_in.reshape(-1)
        buf = buf.cuda()
        assert w.ws_gemm_run(g._h, 0, 0, buf.data_ptr(), 0) == w.WS_OK
        assert g.sync_status() == w.WS_OK
        res = buf.cpu().to(torch.float64).numpy()
        AB, _ = oracle.gemm(np.zeros((M, 0), np.uint16), np.zeros((0, N), np.uint16), "bf16", with_abs=False)
        ref = E.epilogue(AB, C_in.to(torch.float64).numpy(), alpha, beta, out)
        assert compare_exact(res[:M * N].reshape(M, N), ref)["ok"]
        assert np.all(res[M * N:] == SENTINEL)
    finally:
        g.close()


def test_empty_problems_through_the_torch_wrapper():
    g = w.WsGemm(64, 0, 32, (64, 64, 32), 3, 4, 4, "bf16")
    try:
        A = torch.ones((64, 32), dtype=torch.bfloat16, device="cuda")
        B = torch.ones((32, 0), dtype=torch.bfloat16, device="cuda")
        C = g(A, B)
        assert tuple(C.shape) == (64, 0)
    finally:
        g.close()
    g = w.WsGemm(16, 24, 0, (64, 64, 32), 3, 4, 4, "bf16")
    try:
        A = torch.ones((16, 0), dtype=torch.bfloat16, device="cuda")
        B = torch.ones((0, 24), dtype=torch.bfloat16, device="cuda")
        C = g(A, B, torch.full((16, 24), 5.0, device="cuda"))
        assert g.sync_status() == w.WS_OK
        assert bool((C == 0).all())
    finally:
        g.close()


def test_empty_problems_refuse_calibration_and_tracing():
    cfg = w.config((256, 128, 64), 3, 4, 4, "bf16")
    assert w.ws_gemm_create_calibration(0, 256, 256, cfg, w.WS_CALIB_MATH)[0] == w.WS_ERR_UNSUPPORTED
    g = handle(256, 256, 0, ((256, 128, 64), 3, 4, 4))
    try:
        buf = torch.zeros(1 << 12, dtype=torch.int32, device="cuda")
        assert w.ws_gemm_set_trace(g._h, buf.data_ptr(), buf.numel() * 4, 1, 1) == w.WS_ERR_INVALID_ARG
    finally:
        g.close()
