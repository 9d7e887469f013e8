"""Parity of the synchronous (not warp-specialised) baseline kernel with the
CPU oracle: producer_waves = 0, ring depth 1 (load, then multiply) or 2
(double-buffered).  Its 8192^3 sweep points run in test_gpu_parity's
full-size cases."""
import pytest

from paper_2506_11209_amd import inputs
from paper_2506_11209_amd.workloads import WORKLOADS
from tests.gpu_helpers import check_full, log, run_gpu

pytestmark = pytest.mark.gpu

LDS_LIMIT = 163840

SYNC_FAMILIES = []
for dt in ("bf16", "f16"):
    for tk in (32, 64):
        for (tm, tn) in ((32, 32), (64, 64)):
            SYNC_FAMILIES.append(((tm, tn, tk), 1, dt))
        for (tm, tn) in ((64, 64), (64, 128), (128, 64), (128, 128), (128, 256), (256, 128), (256, 256)):
            SYNC_FAMILIES.append(((tm, tn, tk), 4, dt))


def fits(tile, stages):
    tm, tn, tk = tile
    return 256 + stages * 2 * (tm * tk + tk * tn) <= LDS_LIMIT


@pytest.mark.parametrize("stages", [1, 2])
@pytest.mark.parametrize("tile,nc,dtype", SYNC_FAMILIES,
                         ids=lambda x: "x".join(map(str, x)) if isinstance(x, tuple) else str(x))
def test_sync_family_exact_on_integers(tile, nc, dtype, stages):
    if not fits(tile, stages):
        pytest.skip("ring does not fit in LDS")
    tm, tn, tk = tile
    M, N, K = 3 * tm, 5 * tn, 7 * tk
    A, B = inputs.make_operands(M, N, K, dtype, "int4", 300 + tm + tn + tk)
    log("case sync tile=%s nc=%d %s P=%d" % (tile, nc, dtype, stages))
    C = run_gpu(A, B, tile, stages, 0, nc, dtype)
    r = check_full(C, A, B, dtype, exact=True)
    assert r["ok"], r


@pytest.mark.parametrize("stages", [1, 2])
@pytest.mark.parametrize("K", [32, 64, 128, 192])  # S = 1 .. 3 and a tile change inside the prefetch
def test_sync_k_edges(stages, K):
    A, B = inputs.make_operands(256, 512, K, "bf16", "int4", 40 + K)
    log("case sync edges P=%d K=%d" % (stages, K))
    C = run_gpu(A, B, (128, 128, 32), stages, 0, 4, "bf16")
    assert check_full(C, A, B, "bf16", exact=True)["ok"]


def test_sync_multi_round_random_tolerance():
    A, B = inputs.make_operands(2048, 2048, 1024, "bf16", "normal", 43)
    log("case sync multi-round random")
    C = run_gpu(A, B, (256, 256, 64), 2, 0, 4, "bf16")
    r = check_full(C, A, B, "bf16", exact=False)
    assert r["ok"], r
