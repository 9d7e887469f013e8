"""ws_gemm_run_noalloc (the entry point that allocates nothing) against
ws_gemm_create / ws_gemm_run on the same inputs, through the C ABI: its
output must equal the handle path's bit for bit (same kernel, same launch)
and the oracle's (small-integer operands: exact).  Two calls in a row, the
second with a smaller problem, as callers reuse the one static scratch."""
import numpy as np
import pytest
import torch

import oracle
from oracle.check import compare_exact
from paper_2506_11209_amd import inputs
from tests.gpu_helpers import log

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu


def handle_path(M, N, K, cfg, Ad, Bd):
    s, h = w.ws_gemm_create(M, N, K, cfg)
    assert s == w.WS_OK, w.ws_gemm_status_str(s)
    try:
        C = torch.full((M, N), float("nan"), device="cuda")
        st = torch.cuda.current_stream().cuda_stream
        assert w.ws_gemm_run(h, Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(), st) == w.WS_OK
        assert w.ws_gemm_sync_status(h, st) == w.WS_OK
        return C.cpu().numpy()
    finally:
        w.ws_gemm_destroy(h)


def noalloc_path(M, N, K, cfg, Ad, Bd):
    C = torch.full((M, N), float("nan"), device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    s = w.ws_gemm_run_noalloc(M, N, K, cfg, Ad.data_ptr() if Ad is not None else 0,
                              Bd.data_ptr() if Bd is not None else 0, C.data_ptr(), st)
    assert s == w.WS_OK, w.ws_gemm_status_str(s)
    torch.cuda.synchronize()
    return C.cpu().numpy()


# (M, N, K) of the first and the (smaller) second call, tile, stages, np, nc, split
CASES = [
    ((2048, 1024, 1024), (512, 256, 320), (256, 128, 64), 3, 4, 4, 0),
    ((1024, 1024, 768), (256, 512, 256), (256, 256, 64), 2, 4, 8, 1),
    ((1000, 744, 520), (130, 88, 72), (128, 128, 32), 3, 8, 4, 0),  # ragged: general variant
]


@pytest.mark.parametrize("first,second,tile,stages,np_,nc,split", CASES,
                         ids=["256x128x64", "256x256x64-nc8", "ragged-128x128x32"])
def test_noalloc_equals_the_handle_path_twice(first, second, tile, stages, np_, nc, split):
    cfg = w.config(tile, stages, np_, nc, "bf16", "registers", split)
    for i, (M, N, K) in enumerate((first, second)):
        log("case noalloc call %d %dx%dx%d tile=%s nc=%d np=%d" % (i, M, N, K, tile, nc, np_))
        A, B = inputs.make_operands(M, N, K, "bf16", "int4", 60 + i)
        Ad, Bd = A.cuda(), B.cuda()
        C0 = noalloc_path(M, N, K, cfg, Ad, Bd)
        C1 = handle_path(M, N, K, cfg, Ad, Bd)
        assert np.array_equal(C0.view(np.uint32), C1.view(np.uint32))
        ref, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), "bf16", with_abs=False)
        r = compare_exact(C0, ref)
        assert r["ok"], r


def test_noalloc_random_values_match_the_handle_path():
    M, N, K = 1024, 768, 2048
    cfg = w.config((128, 128, 64), 4, 4, 4, "bf16")
    A, B = inputs.make_operands(M, N, K, "bf16", "normal", 61)
    Ad, Bd = A.cuda(), B.cuda()
    log("case noalloc random")
    C0 = noalloc_path(M, N, K, cfg, Ad, Bd)
    C1 = handle_path(M, N, K, cfg, Ad, Bd)
    assert np.array_equal(C0.view(np.uint32), C1.view(np.uint32))


def test_noalloc_empty_and_k0_and_rejections():
    cfg = w.config((128, 128, 64), 3, 4, 4, "bf16")
    st = torch.cuda.current_stream().cuda_stream
    assert w.ws_gemm_run_noalloc(0, 64, 64, cfg, 0, 0, 0, st) == w.WS_OK       # nothing to do
    C = noalloc_path(96, 40, 0, cfg, None, None)                                # K = 0: zeros
    assert np.all(C == 0.0)
    buf = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    p = buf.data_ptr()
    assert w.ws_gemm_run_noalloc(128, 128, 128, cfg, p + 2, p, p, st) == w.WS_ERR_INVALID_ARG
    assert w.ws_gemm_run_noalloc(128, 128, 128, cfg, 0, p, p, st) == w.WS_ERR_INVALID_ARG
    bad = w.config((128, 128, 64), 9, 4, 4, "bf16")
    assert w.ws_gemm_run_noalloc(128, 128, 128, bad, p, p, p, st) == w.WS_ERR_INVALID_ARG
    torch.cuda.synchronize()
