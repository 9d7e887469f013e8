"""Shapes the tiles do not divide (the ragged kernel variant): partial edge
tiles in M and N, a partial last K-iteration, and nothing written outside C.
Checked against the CPU oracle over all of C."""
import numpy as np
import pytest
import torch

from paper_2506_11209_amd import inputs
from tests.gpu_helpers import check_full, log

pytestmark = pytest.mark.gpu

SHAPES = [(1, 8, 8), (7, 136, 72), (129, 264, 200), (300, 520, 4104), (257, 8, 4104), (1000, 1000, 1000)]
CONFIGS = [((256, 128, 64), 3, 4, 4), ((128, 256, 32), 4, 8, 4), ((64, 64, 64), 3, 4, 4),
           ((32, 32, 32), 2, 1, 1), ((64, 64, 32), 3, 2, 1), ((256, 128, 64), 3, 8, 4),
           ((256, 256, 64), 2, 4, 8)]
GUARD = 4096
SENTINEL = -7.0


def run_ragged(A, B, tile, stages, np_, nc, dtype, load_path="registers"):
    from paper_2506_11209_amd import wsgemm as w
    M, K = A.shape
    N = B.shape[1]
    g = w.WsGemm(M, N, K, tile, stages, np_, nc, dtype, load_path)
    try:
        assert g.info.ragged == 1
        buf = torch.full((M * N + GUARD,), SENTINEL, dtype=torch.float32, device="cuda")
        C = buf[:M * N].view(M, N)
        Ad, Bd = A.cuda(), B.cuda()  # held until the kernel has finished
        g.run_ptrs(Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(), torch.cuda.current_stream().cuda_stream)
        assert g.sync_status() == w.WS_OK
        out = buf.cpu().numpy()
        return out[:M * N].reshape(M, N), out[M * N:]
    finally:
        g.close()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("tile,stages,np_,nc", CONFIGS, ids=lambda x: "x".join(map(str, x)) if isinstance(x, tuple) else str(x))
@pytest.mark.parametrize("M,N,K", SHAPES, ids=lambda x: str(x))
def test_ragged_exact_on_integers(M, N, K, tile, stages, np_, nc, dtype):
    if M % tile[0] == 0 and N % tile[1] == 0 and K % tile[2] == 0:
        pytest.skip("whole tiles")
    A, B = inputs.make_operands(M, N, K, dtype, "int4", 500 + M + N + K)
    log("case ragged %dx%dx%d tile=%s %d:%d %s" % (M, N, K, tile, np_, nc, dtype))
    C, guard = run_ragged(A, B, tile, stages, np_, nc, dtype)
    assert np.all(guard == SENTINEL), "wrote past the end of C"
    r = check_full(C, A, B, dtype, exact=True)
    assert r["ok"], r


@pytest.mark.parametrize("load_path", ["registers", "dma"])
def test_ragged_random_within_tolerance(load_path):
    # the ragged variant always loads through registers, whatever load_path says
    A, B = inputs.make_operands(1000, 1000, 1000, "bf16", "normal", 77)
    log("case ragged random %s" % load_path)
    C, guard = run_ragged(A, B, (256, 128, 64), 3, 4, 4, "bf16", load_path)
    assert np.all(guard == SENTINEL)
    r = check_full(C, A, B, "bf16", exact=False)
    assert r["ok"], r
