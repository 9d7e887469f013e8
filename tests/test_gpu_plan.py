"""The host planner's occupancy (LDS, waves and the compiled kernel's
registers, no GPU) agrees with the runtime's occupancy query that
ws_gemm_create uses, for every compiled GEMM configuration."""
import pytest

from paper_2506_11209_amd.build import MODE_GEMM, instances

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu

LDS_LIMIT = 163840


def configs():
    out = set()
    for (tm, tn, tk, nc, np_, split, bf16, trace, mode, ragged) in instances():
        if trace or ragged or mode != MODE_GEMM:
            continue
        for P in ((1, 2) if np_ == 0 else (2, 3, 4, 6)):
            if 256 + P * 2 * (tm * tk + tk * tn) <= LDS_LIMIT:
                out.add(((tm, tn, tk), P, np_, nc, split, "bf16" if bf16 else "f16"))
    return sorted(out)


def test_planned_occupancy_matches_the_runtime():
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    bad = []
    for tile, P, np_, nc, split, dt in configs():
        M, N, K = 64 * tile[0], 64 * tile[1], 2 * tile[2]  # enough tiles to fill every slot
        cfg = w.config(tile, P, np_, nc, dt, split=split)
        s, planned = w.ws_gemm_plan(M, N, K, cfg, cus, 0)
        assert s == w.WS_OK
        g = w.WsGemm(M, N, K, tile, P, np_, nc, dt, split=split)
        try:
            if g.info.grid != planned.grid:
                bad.append((tile, P, np_, nc, split, dt, planned.grid // cus, g.info.grid // cus))
        finally:
            g.close()
    assert not bad, "planned vs runtime workgroups per CU: %s" % bad
