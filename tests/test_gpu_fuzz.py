"""Seeded random cases over every compiled specialised configuration: random
shapes (whole or ragged tiles, down to a single row), ring depths, load paths
and epilogues, on small-integer operands so that every case must match the
oracle bit for bit.  Each case prints its parameters before it runs."""
import numpy as np
import pytest
import torch

import oracle
from oracle import epilogue_ref as E
from oracle.check import compare_exact
from paper_2506_11209_amd import inputs
from paper_2506_11209_amd.build import MODE_GEMM, instances
from tests.gpu_helpers import log

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu

GUARD = 512
SENTINEL = -7.0
TORCH_OUT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
CONFIGS = sorted({(tm, tn, tk, nc, np_, split, bf16)
                  for (tm, tn, tk, nc, np_, split, bf16, trace, mode, general) in instances()
                  if np_ > 0 and mode == MODE_GEMM and not trace})
N_CASES = 400


def draw_case(i):
    rng = np.random.default_rng(7000 + i)
    tm, tn, tk, nc, np_, split, bf16 = CONFIGS[i % len(CONFIGS)]
    dtype = "bf16" if bf16 else "f16"
    if rng.random() < 0.3:  # whole tiles
        M, N, K = (int(rng.integers(1, 4)) * tm, int(rng.integers(1, 4)) * tn, int(rng.integers(1, 5)) * tk)
    else:                   # ragged: any M, N and K multiples of 8
        M = int(rng.integers(1, 3 * tm + 1))
        N = 8 * int(rng.integers(1, (3 * tn) // 8 + 1))
        K = 8 * int(rng.integers(1, (4 * tk) // 8 + 1))
    max_stages = max(2, min(8, (163840 - 256) // (2 * (tm * tk + tk * tn))))
    stages = int(rng.integers(2, max_stages + 1))
    load_path = "dma" if rng.random() < 0.5 else "registers"
    if rng.random() < 0.5:
        epi = (1.0, 0.0, "f32")
    else:
        epi = (float(rng.choice([1.0, 0.5, -2.0, 0.25])), float(rng.choice([0.0, 1.0, -0.5, 2.0])),
               str(rng.choice(["f32", "bf16", "f16"])))
    return dict(M=M, N=N, K=K, tile=(tm, tn, tk), stages=stages, np_=np_, nc=nc, split=split,
                dtype=dtype, load_path=load_path, epi=epi, seed=8000 + i)


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_case_is_exact(i):
    c = draw_case(i)
    log("case fuzz %d %s" % (i, c))
    M, N, K = c["M"], c["N"], c["K"]
    alpha, beta, out = c["epi"]
    A, B = inputs.make_operands(M, N, K, c["dtype"], "int4", c["seed"])
    C_in = inputs.make_output(M, N, out, "int4", c["seed"] + 1)
    g = w.WsGemm(M, N, K, c["tile"], c["stages"], c["np_"], c["nc"], c["dtype"], c["load_path"],
                 split=c["split"])
    try:
        g.set_epilogue(alpha, beta, out)
        buf = torch.full((M * N + GUARD,), SENTINEL, dtype=TORCH_OUT[out])
        buf[:M * N] = C_in.reshape(-1)
        buf = buf.cuda()
        Ad, Bd = A.cuda(), B.cuda()
        g.run_ptrs(Ad.data_ptr(), Bd.data_ptr(), buf.data_ptr(), torch.cuda.current_stream().cuda_stream)
        assert g.sync_status() == w.WS_OK
        res = buf.cpu().to(torch.float64).numpy()
    finally:
        g.close()
    assert np.all(res[M * N:] == SENTINEL), "wrote past the end of C"
    AB, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), c["dtype"], with_abs=False)
    ref = E.epilogue(AB, C_in.to(torch.float64).numpy(), alpha, beta, out)
    r = compare_exact(res[:M * N].reshape(M, N), ref)
    assert r["ok"], (c, r)


SYNC_CONFIGS = sorted({(tm, tn, tk, nc, bf16)
                       for (tm, tn, tk, nc, np_, split, bf16, trace, mode, general) in instances() if np_ == 0})
N_SYNC_CASES = 2 * len(SYNC_CONFIGS)


@pytest.mark.parametrize("i", range(N_SYNC_CASES))
def test_random_synchronous_case_is_exact(i):
    """The synchronous kernel (no producer waves) takes whole tiles and the
    default epilogue: random multiples of each compiled tile, ring depth 1
    or 2 where it fits."""
    rng = np.random.default_rng(9000 + i)
    tm, tn, tk, nc, bf16 = SYNC_CONFIGS[i % len(SYNC_CONFIGS)]
    dtype = "bf16" if bf16 else "f16"
    M, N, K = (int(rng.integers(1, 4)) * tm, int(rng.integers(1, 4)) * tn, int(rng.integers(1, 6)) * tk)
    fits2 = 256 + 2 * 2 * (tm * tk + tk * tn) <= 163840
    stages = int(rng.integers(1, 3)) if fits2 else 1
    log("case fuzz sync %d %dx%dx%d tile=%s nc=%d P=%d %s" % (i, M, N, K, (tm, tn, tk), nc, stages, dtype))
    A, B = inputs.make_operands(M, N, K, dtype, "int4", 9500 + i)
    g = w.WsGemm(M, N, K, (tm, tn, tk), stages, 0, nc, dtype)
    try:
        buf = torch.full((M * N + GUARD,), SENTINEL, device="cuda")
        Ad, Bd = A.cuda(), B.cuda()
        g.run_ptrs(Ad.data_ptr(), Bd.data_ptr(), buf.data_ptr(), torch.cuda.current_stream().cuda_stream)
        assert g.sync_status() == w.WS_OK
        res = buf.cpu().numpy()
    finally:
        g.close()
    assert np.all(res[M * N:] == SENTINEL)
    AB, _ = oracle.gemm(inputs.bits(A), inputs.bits(B), dtype, with_abs=False)
    r = compare_exact(res[:M * N].reshape(M, N), AB)
    assert r["ok"], r
