"""Epilogue variants (ws_gemm_set_epilogue): C <- alpha (A B) + beta C stored
as f32, bf16 or f16, on whole and partial tiles, checked against the CPU
oracle (the exact product from the GEMM oracle, the epilogue and its one
rounding from oracle/epilogue_ref.py).

Exact cases use small integers with power-of-two alpha and beta: every
binary32 step is then exact, so the GPU and the oracle round the same value
once and must agree bit for bit.  Random cases use the accumulation bound
plus one rounding of the output type."""
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

GUARD = 2048
SENTINEL = -7.0
TORCH_OUT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}

# (M, N, K), tile, stages, producer waves, consumer waves, input dtype
LAUNCHES = [
    ((256, 256, 128), (128, 128, 32), 3, 4, 4, "bf16"),    # whole tiles, 1:1
    ((256, 512, 256), (256, 128, 64), 3, 8, 4, "bf16"),    # whole tiles, 2:1 (single-buffered consumer)
    ((129, 264, 200), (256, 128, 64), 3, 4, 4, "bf16"),    # partial tiles in M, N and K
    ((300, 136, 72), (64, 64, 32), 3, 2, 1, "f16"),        # partial tiles, one consumer wave, 2:1
    ((512, 256, 192), (256, 256, 64), 2, 4, 8, "bf16"),    # whole tiles, eight consumer waves (roll loop)
    ((300, 264, 200), (256, 256, 64), 2, 4, 8, "bf16"),    # partial tiles, eight consumer waves
]
COEFFS = [(1.0, 0.0), (0.5, 0.0), (-2.0, 1.0), (0.5, -0.25), (0.0, 1.0)]


def run_epilogue(A, B, C_in, launch, alpha, beta, out):
    (M, N, K), tile, stages, np_, nc, dtype = launch
    g = w.WsGemm(M, N, K, tile, stages, np_, nc, dtype)
    try:
        g.set_epilogue(alpha, beta, out)
        # the default epilogue keeps the plain kernel on whole tiles
        default = (alpha, beta, out) == (1.0, 0.0, "f32")
        assert g.info.general == (0 if default and not g.info.ragged else 1)
        buf = torch.full((M * N + GUARD,), SENTINEL, dtype=TORCH_OUT[out])
        buf[:M * N] = C_in.reshape(-1)
        buf = buf.cuda()
        Ad, Bd = A.cuda(), B.cuda()
        g.run_ptrs(Ad.data_ptr(), Bd.data_ptr(), buf.data_ptr(), torch.cuda.current_stream().cuda_stream)
        assert g.sync_status() == w.WS_OK
        res = buf.cpu().to(torch.float64).numpy()
        return res[:M * N].reshape(M, N), res[M * N:]
    finally:
        g.close()


def _id(x):
    return "x".join(map(str, x)) if isinstance(x, tuple) else str(x)


@pytest.mark.parametrize("out", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("alpha,beta", COEFFS, ids=lambda c: str(c))
@pytest.mark.parametrize("launch", LAUNCHES, ids=lambda l: "%s-%s-%d-%d" % (_id(l[0]), _id(l[1]), l[3], l[4]))
def test_epilogue_exact_on_integers(launch, alpha, beta, out):
    (M, N, K), _, _, _, _, dtype = launch
    A, B = inputs.make_operands(M, N, K, dtype, "int4", 900 + M + K)
    C_in = inputs.make_output(M, N, out, "int4", 901 + N)
    log("case epilogue %s alpha=%g beta=%g out=%s" % (launch, alpha, beta, out))
    C, guard = run_epilogue(A, B, C_in, launch, alpha, beta, out)
    assert np.all(guard == SENTINEL), "wrote past the end of C"
    AB, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), dtype, with_abs=False)
    ref = E.epilogue(AB, C_in.to(torch.float64).numpy(), alpha, beta, out)
    r = compare_exact(C, ref)
    assert r["ok"], r


@pytest.mark.parametrize("out", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("launch", [LAUNCHES[1], ((1000, 1000, 1000), (256, 128, 64), 3, 4, 4, "bf16")],
                         ids=["whole", "ragged"])
def test_epilogue_random_within_tolerance(launch, out):
    (M, N, K), _, _, _, _, dtype = launch
    alpha, beta = 1.5, -0.75
    A, B = inputs.make_operands(M, N, K, dtype, "normal", 31 + K)
    C_in = inputs.make_output(M, N, out, "normal", 32)
    log("case epilogue random %s out=%s" % (launch, out))
    C, guard = run_epilogue(A, B, C_in, launch, alpha, beta, out)
    assert np.all(guard == SENTINEL)
    AB, S = oracle.gemm(inputs.bits(A), inputs.bits(B), dtype)
    c_in = C_in.to(torch.float64).numpy()
    exact = float(np.float32(alpha)) * AB + float(np.float32(beta)) * c_in
    bound = E.epilogue_bound(S, c_in, alpha, beta, exact, out)
    err = np.abs(C - exact)
    assert np.all(np.isfinite(C))
    assert np.all(err <= bound), float(np.max(err / bound))


def test_beta_zero_does_not_read_c():
    launch = LAUNCHES[2]
    (M, N, K), _, _, _, _, dtype = launch
    A, B = inputs.make_operands(M, N, K, dtype, "int4", 5)
    C_in = torch.full((M, N), float("nan"), dtype=torch.bfloat16)
    C, _ = run_epilogue(A, B, C_in, launch, 2.0, 0.0, "bf16")
    AB, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), dtype, with_abs=False)
    r = compare_exact(C, E.epilogue(AB, None, 2.0, 0.0, "bf16"))
    assert r["ok"], r


def test_f16_overflow_gives_infinity():
    launch = LAUNCHES[0]
    (M, N, K), _, _, _, _, dtype = launch
    A, B = inputs.make_operands(M, N, K, dtype, "int4", 8)
    C_in = inputs.make_output(M, N, "f16", "int4", 9)
    alpha = 2.0**12
    C, _ = run_epilogue(A, B, C_in, launch, alpha, 1.0, "f16")
    AB, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), dtype, with_abs=False)
    ref = E.epilogue(AB, C_in.to(torch.float64).numpy(), alpha, 1.0, "f16")
    assert np.isinf(ref).any() and np.isfinite(ref).any()
    r = compare_exact(C, ref)
    assert r["ok"], r


def test_default_epilogue_restores_the_plain_kernel():
    M = N = K = 512
    A, B = inputs.make_operands(M, N, K, "bf16", "int4", 11)
    g = w.WsGemm(M, N, K, (128, 128, 32), 3, 4, 4, "bf16")
    try:
        plain = g.info.as_dict()
        assert plain["general"] == 0
        g.set_epilogue(1.0, 0.0, "bf16")
        assert g.info.general == 1
        g.set_epilogue()  # the default: C = A B in fp32
        assert g.info.as_dict() == plain
        C = g(A.cuda(), B.cuda())
        assert g.sync_status() == w.WS_OK
        AB, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), "bf16", with_abs=False)
        assert compare_exact(C.cpu().numpy(), AB)["ok"]
    finally:
        g.close()


def test_epilogue_and_tracing_exclude_each_other():
    g = w.WsGemm(512, 512, 512, (128, 128, 32), 3, 4, 4, "bf16")
    buf = torch.zeros(1 << 16, dtype=torch.int32, device="cuda")
    try:
        g.set_epilogue(0.5, 0.0, "f32")
        s = w.library().ws_gemm_set_trace(g._h, w._p(buf.data_ptr()), buf.numel() * 4, 1, 4)
        assert s == w.WS_ERR_UNSUPPORTED
        g.set_epilogue()
        assert w.library().ws_gemm_set_trace(g._h, w._p(buf.data_ptr()), buf.numel() * 4, 1, 4) == w.WS_OK
        epi = w.ws_gemm_epilogue(0.5, 0.0, w.WS_OUT_F32)
        assert w.ws_gemm_set_epilogue(g._h, epi) == w.WS_ERR_UNSUPPORTED
    finally:
        g.close()


def test_epilogue_rejections():
    g = w.WsGemm(512, 512, 512, (128, 128, 32), 2, 0, 4, "bf16")  # synchronous kernel
    try:
        assert w.ws_gemm_set_epilogue(g._h, w.ws_gemm_epilogue(2.0, 0.0, w.WS_OUT_F32)) == w.WS_ERR_UNSUPPORTED
        assert w.ws_gemm_set_epilogue(g._h, None) == w.WS_OK
    finally:
        g.close()
    g = w.WsGemm(512, 512, 512, (128, 128, 64), 3, 4, 4, "bf16", calibration="math")
    try:
        assert w.ws_gemm_set_epilogue(g._h, w.ws_gemm_epilogue(1.0, 1.0, w.WS_OUT_F32)) == w.WS_ERR_UNSUPPORTED
    finally:
        g.close()
    g = w.WsGemm(512, 512, 512, (128, 128, 32), 3, 4, 4, "bf16")
    try:
        for epi in (w.ws_gemm_epilogue(float("nan"), 0.0, 0), w.ws_gemm_epilogue(1.0, float("inf"), 0),
                    w.ws_gemm_epilogue(1.0, 0.0, 3), w.ws_gemm_epilogue(1.0, 0.0, -1)):
            assert w.ws_gemm_set_epilogue(g._h, epi) == w.WS_ERR_INVALID_ARG
        # a 16-bit C needs only 2-byte alignment; fp32 keeps 4
        g.set_epilogue(1.0, 0.0, "bf16")
        A = torch.zeros(512 * 512 + 8, dtype=torch.bfloat16, device="cuda")
        C = torch.zeros(512 * 512 + 8, dtype=torch.bfloat16, device="cuda")
        assert w.ws_gemm_run(g._h, A.data_ptr(), A.data_ptr(), C.data_ptr() + 2, 0) == w.WS_OK
        g.set_epilogue()
        assert w.ws_gemm_run(g._h, A.data_ptr(), A.data_ptr(), C.data_ptr() + 2, 0) == w.WS_ERR_INVALID_ARG
        torch.cuda.synchronize()
    finally:
        g.close()
