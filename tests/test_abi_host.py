"""C-ABI host logic: symbols, validation, planning and the tile schedule (no GPU)."""
import os
import re

import pytest

from paper_2506_11209_amd import wsgemm as w
from paper_2506_11209_amd.workloads import WORKLOADS, split_of, unpack

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def declared_functions():
    """Every function declared in the public headers include/*.h."""
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(ws_\w+)\s*\(", text))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 11 and "ws_model_predict" in names
    lib = w.library()
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_abi_version_and_status_text():
    assert w.ws_gemm_abi_version() == 7
    for s in range(7):
        assert w.ws_gemm_status_str(s) and w.ws_gemm_status_str(s) != "unknown status"
    assert w.ws_gemm_status_str(99) == "unknown status"


def cfg(tile=(256, 128, 64), stages=3, np_=4, nc=4, dtype="bf16"):
    return w.config(tile, stages, np_, nc, dtype)


def test_plan_headline_shape():
    s, info = w.ws_gemm_plan(8192, 8192, 8192, cfg(), 256, 1)
    assert s == w.WS_OK
    d = info.as_dict()
    assert d["tiles"] == 32 * 64 and d["grid"] == 256 and d["rounds"] == 8 and d["iters"] == 128
    assert d["block"] == 512 and d["split"] == 1 and d["xcd_remap"] == 1
    assert d["lds_bytes"] == 256 + 3 * 2 * (256 * 64 + 64 * 128)


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_plan_every_workload_point(name):
    wl = WORKLOADS[name]
    for pt in wl.points:
        tm, tn, tk, stages, np_, nc, split = unpack(pt)
        c = cfg((tm, tn, tk), stages, np_, nc, wl.dtype)
        c.split = split
        s, info = w.ws_gemm_plan(wl.M, wl.N, wl.K, c, 256, 1)
        stage = 2 * (tm * tk + tk * tn)
        if 256 + stages * stage > 163840:
            assert s == w.WS_ERR_LDS_OVERFLOW
            continue
        assert s == w.WS_OK, (name, tm, tn, tk, stages, np_, nc, w.ws_gemm_status_str(s))
        tiles = (wl.M // tm) * (wl.N // tn)
        assert info.tiles == tiles and info.iters == wl.K // tk
        assert info.grid == min(tiles, 256)
        assert info.rounds == -(-tiles // info.grid)
        assert info.split == split_of(pt) and info.block == 64 * (np_ + nc)


@pytest.mark.parametrize("tiles_m,tiles_n,resident,expect_per_cu", [
    (64, 64, 5, 4),   # 4096 tiles: four rounds of four beat four rounds of five
    (80, 64, 5, 5),   # 5120 tiles: four rounds of five fill every slot
    (32, 32, 3, 2),   # 1024 tiles: 2 rounds of 2 (4) against 2 of 3 (6); 1 x 4 ties, the larger wins
    (32, 32, 4, 4),   # 1024 tiles: one round of four
    (1, 100, 4, 1),   # 100 tiles: fewer tiles than CUs
])
def test_grid_balances_rounds_against_sharing(tiles_m, tiles_n, resident, expect_per_cu):
    # the synchronous kernel (128 x 128 x 32, ring depth 1) with the given
    # resident workgroups per CU on 256 CUs
    c = cfg((128, 128, 32), 1, 0, 4, "bf16")
    s, info = w.ws_gemm_plan(128 * tiles_m, 128 * tiles_n, 64, c, 256, resident)
    assert s == w.WS_OK
    tiles = tiles_m * tiles_n
    assert info.grid == min(tiles, 256 * expect_per_cu)
    assert info.rounds == -(-tiles // info.grid)
    # no other count of workgroups per CU costs fewer rounds x workgroups per CU
    cost = lambda u: -(-tiles // (256 * u)) * u
    assert all(cost(u) >= cost(expect_per_cu) for u in range(1, resident + 1))


def test_lds_overflow_case_from_the_sweep():
    # (256,128,64) x 4 stages = 192 KiB + header > 160 KiB
    s, _ = w.ws_gemm_plan(8192, 8192, 8192, cfg((256, 128, 64), 4), 256, 1)
    assert s == w.WS_ERR_LDS_OVERFLOW


@pytest.mark.parametrize("M,N,K,tile,status", [
    (8192, 8192, 8192 + 4, (256, 128, 64), w.WS_ERR_NOT_DIVISIBLE),   # ragged K not a multiple of 8
    (8192, 8192 + 12, 8192, (256, 128, 64), w.WS_ERR_NOT_DIVISIBLE),  # ragged N not a multiple of 8
    (-1, 8192, 8192, (256, 128, 64), w.WS_ERR_INVALID_ARG),
    (8192, -1, 8192, (256, 128, 64), w.WS_ERR_INVALID_ARG),
    (8192, 8192, -8, (256, 128, 64), w.WS_ERR_INVALID_ARG),
    (0, 8192, 8192, (48, 128, 64), w.WS_ERR_INVALID_ARG),           # empty, but a bad tile
    (0, 8192, 8192, (256, 256, 32), w.WS_ERR_UNSUPPORTED),          # empty, unsupported waves
    (8192, 8192, 0, (256, 128, 128), w.WS_ERR_LDS_OVERFLOW),        # empty, ring too large
    (8192, 8192, 8192, (48, 128, 64), w.WS_ERR_INVALID_ARG),
    (8192, 8192, 8192, (512, 128, 64), w.WS_ERR_INVALID_ARG),
    (8192, 8192, 8192, (256, 128, 16), w.WS_ERR_INVALID_ARG),
    (8192, 8192, 8192, (256, 256, 32), w.WS_ERR_UNSUPPORTED),  # 128x128 wave tile
])
def test_plan_rejections(M, N, K, tile, status):
    s, _ = w.ws_gemm_plan(M, N, K, cfg(tile), 256, 1)
    assert s == status, w.ws_gemm_status_str(s)


@pytest.mark.parametrize("np_,nc,stages,status", [
    (3, 4, 3, w.WS_ERR_UNSUPPORTED), (4, 2, 3, w.WS_ERR_UNSUPPORTED), (4, 4, 1, w.WS_ERR_INVALID_ARG),
    (4, 4, 9, w.WS_ERR_INVALID_ARG), (16, 4, 2, w.WS_ERR_UNSUPPORTED), (8, 8, 2, w.WS_ERR_UNSUPPORTED),
    (2, 8, 2, w.WS_ERR_UNSUPPORTED),
])
def test_plan_rejects_wave_and_stage_counts(np_, nc, stages, status):
    s, _ = w.ws_gemm_plan(4096, 4096, 4096, cfg((128, 128, 32), stages, np_, nc), 256, 1)
    assert s == status


@pytest.mark.parametrize("np_,nc,split,want", [
    (4, 4, 0, 1), (8, 4, 0, 2), (4, 4, 1, 1), (4, 4, 2, 2), (8, 4, 2, 2), (1, 1, 0, 1), (2, 1, 0, 2),
    (4, 8, 0, 1), (4, 8, 1, 1), (4, 8, 2, 2),
    (8, 4, 1, None), (1, 1, 2, None), (2, 1, 1, None), (0, 4, 1, None), (4, 4, 3, "invalid"),
])
def test_plan_split_of_each_arrangement(np_, nc, split, want):
    """split 0 derives the arrangement from the wave counts; an explicit one
    must be an arrangement some kernel has."""
    tile = (256, 256, 64) if nc == 8 else (128, 128, 64) if nc == 4 else (64, 64, 64)
    c = cfg(tile, 2, np_, nc)
    c.split = split
    s, info = w.ws_gemm_plan(4096, 4096, 4096, c, 256, 1)
    if want == "invalid":
        assert s == w.WS_ERR_INVALID_ARG
    elif want is None:
        assert s == w.WS_ERR_UNSUPPORTED
    else:
        assert s == w.WS_OK and info.split == want and info.block == 64 * (np_ + nc)


def test_plan_bad_dtype_and_cus():
    c = cfg()
    c.dtype = 7
    assert w.ws_gemm_plan(8192, 8192, 8192, c, 256, 1)[0] == w.WS_ERR_INVALID_ARG
    assert w.ws_gemm_plan(8192, 8192, 8192, cfg(), 0, 1)[0] == w.WS_ERR_INVALID_ARG


def test_null_handles_are_rejected():
    assert w.ws_gemm_destroy(None) == w.WS_OK
    assert w.ws_gemm_run(None, 16, 16, 16, 0) == w.WS_ERR_INVALID_ARG
    assert w.ws_gemm_sync_status(None, 0) == w.WS_ERR_INVALID_ARG
    assert w.ws_gemm_query(None)[0] == w.WS_ERR_INVALID_ARG
    assert w.ws_gemm_set_debug(None, None) == w.WS_ERR_INVALID_ARG
    assert w.ws_gemm_set_epilogue(None, None) == w.WS_ERR_INVALID_ARG
    assert w.ws_gemm_set_epilogue(None, w.ws_gemm_epilogue(2.0, 1.0, w.WS_OUT_BF16)) == w.WS_ERR_INVALID_ARG


def _schedule(info):
    seen = {}
    for r in range(info.rounds + 1):
        for g in range(info.grid):
            s, ti, tj = w.ws_gemm_schedule(info, g, r)
            if s == w.WS_OK:
                assert (ti, tj) not in seen, "tile computed twice"
                seen[(ti, tj)] = (g, r)
            else:
                assert r * info.grid + g >= info.tiles or r == info.rounds
    return seen


@pytest.mark.parametrize("shape,tile,cus", [
    ((8192, 8192), (256, 128, 64), 256), ((4096, 4096), (128, 128, 32), 256),
    ((16384, 256), (128, 64, 64), 256), ((2048, 2048), (128, 128, 64), 256),
    ((1024, 3072), (64, 64, 32), 84), ((640, 448), (64, 64, 32), 100),
])
def test_schedule_covers_every_tile_once(shape, tile, cus):
    M, N = shape
    s, info = w.ws_gemm_plan(M, N, 1024, cfg(tile, 2), cus, 1)
    assert s == w.WS_OK
    seen = _schedule(info)
    assert len(seen) == info.tiles
    assert {k for k in seen} == {(i, j) for i in range(info.tiles_m) for j in range(info.tiles_n)}


def test_xcd_blocks_are_compact():
    """Tiles running together on one XCD form a group_m x (32/group_m) block."""
    s, info = w.ws_gemm_plan(8192, 8192, 8192, cfg(), 256, 1)
    for r in range(info.rounds):
        for x in range(8):
            tiles = [w.ws_gemm_schedule(info, g, r)[1:] for g in range(x, 256, 8)]
            rows = {t[0] for t in tiles}
            cols = {t[1] for t in tiles}
            assert len(rows) * len(cols) == 32 and len(rows) == info.group_m


def test_paper_wave_example():
    """Section 2.1: 256 output tiles on 84 SMs take four waves; 80 SMs get
    three tiles and four SMs get four (tests/golden/paper_wave_example.txt)."""
    vals = {}
    for line in open(os.path.join(GOLDEN, "paper_wave_example.txt")):
        line = line.split("#")[0].strip()
        if line:
            k, v = line.split("=")
            vals[k.strip()] = int(v)
    # 256 tiles of 64x64 on a 1024x1024 output, one workgroup per SM
    s, info = w.ws_gemm_plan(1024, 1024, 256, cfg((64, 64, 32), 2, 1, 1), vals["sms"], 1)
    assert s == w.WS_OK and info.tiles == vals["tiles"] and info.grid == vals["sms"]
    assert info.rounds == vals["waves"]
    seen = _schedule(info)
    per_wg = {}
    for (g, r) in seen.values():
        per_wg[g] = per_wg.get(g, 0) + 1
    counts = sorted(per_wg.values())
    assert counts.count(3) == vals["sms_with_3"] and counts.count(4) == vals["sms_with_4"]


def test_calibration_kind_is_validated_before_the_device():
    for kind in (-2, -1, 6, 99):
        s, h = w.ws_gemm_create_calibration(256, 256, 256, cfg((64, 64, 64), 2), kind)
        assert s == w.WS_ERR_INVALID_ARG and not h.value


def test_calibration_needs_a_compiled_variant():
    # calibration kernels exist for bf16 configurations with four consumer waves
    s, h = w.ws_gemm_create_calibration(256, 256, 256, cfg((64, 64, 64), 2, dtype="f16"),
                                        w.WS_CALIB_MATH)
    assert s == w.WS_ERR_UNSUPPORTED and not h.value
    s, h = w.ws_gemm_create_calibration(256, 256, 256, cfg((32, 32, 32), 2, 1, 1), w.WS_CALIB_LOAD_A)
    assert s == w.WS_ERR_UNSUPPORTED and not h.value


def test_plan_synchronous_kernel():
    # producer_waves = 0: every wave loads and computes; ring depth 1 or 2
    for P in (1, 2):
        s, info = w.ws_gemm_plan(8192, 8192, 8192, cfg((256, 256, 64), P, 0, 4), 256, 1)
        assert s == w.WS_OK and info.split == 0 and info.block == 256
        assert info.lds_bytes == 256 + P * 2 * (256 * 64 + 64 * 256)
    assert w.ws_gemm_plan(8192, 8192, 8192, cfg((256, 256, 64), 3, 0, 4), 256, 1)[0] == w.WS_ERR_INVALID_ARG
    # 128 x 128 wave tiles only without producer waves
    assert w.ws_gemm_plan(8192, 8192, 8192, cfg((256, 256, 32), 2, 4, 4), 256, 1)[0] == w.WS_ERR_UNSUPPORTED
    assert w.ws_gemm_plan(1024, 1024, 1024, cfg((128, 128, 32), 1, 0, 4), 256, 1)[0] == w.WS_OK


@pytest.mark.parametrize("M,N,K", [(8192, 8192, 8192 + 32), (8192 + 64, 8192, 8192), (8192, 8192 + 32, 8192),
                                   (1, 8, 8), (1000, 136, 72), (257, 8, 4104)])
def test_plan_ragged_shapes(M, N, K):
    tm, tn, tk = 256, 128, 64
    s, info = w.ws_gemm_plan(M, N, K, cfg((tm, tn, tk)), 256, 1)
    assert s == w.WS_OK and info.ragged == 1 and info.general == 1
    assert info.tiles_m == -(-M // tm) and info.tiles_n == -(-N // tn) and info.iters == -(-K // tk)
    # whole tiles are not ragged
    s, info = w.ws_gemm_plan(8192, 8192, 8192, cfg((tm, tn, tk)), 256, 1)
    assert info.ragged == 0 and info.general == 0
    # the synchronous kernel takes whole tiles only
    assert w.ws_gemm_plan(M, N, K, cfg((tm, tn, tk), 2, 0, 4), 256, 1)[0] == w.WS_ERR_NOT_DIVISIBLE


@pytest.mark.parametrize("M,N,K", [(0, 8192, 8192), (8192, 0, 8192), (8192, 8192, 0), (0, 0, 0), (5, 12, 0)])
def test_plan_empty_problems(M, N, K):
    """Empty problems plan no GEMM launch (grid 0); the configuration is
    still validated, and shapes the tiles would not divide are accepted
    (there is nothing to tile)."""
    tm, tn, tk = 256, 128, 64
    s, info = w.ws_gemm_plan(M, N, K, cfg((tm, tn, tk)), 256, 1)
    assert s == w.WS_OK, w.ws_gemm_status_str(s)
    assert info.grid == 0 and info.tiles == 0 and info.rounds == 0 and info.ragged == 0
    assert info.tiles_m == -(-M // tm) and info.tiles_n == -(-N // tn) and info.iters == -(-K // tk)
    assert info.block == 512 and info.lds_bytes == 256 + 3 * 2 * (tm * tk + tk * tn)
    # no tile to schedule
    assert w.ws_gemm_schedule(info, 0, 0)[0] == w.WS_ERR_INVALID_ARG
    # the synchronous kernel's configurations plan empty problems too
    assert w.ws_gemm_plan(M, N, K, cfg((tm, tn, tk), 2, 0, 4), 256, 1)[0] == w.WS_OK



@pytest.mark.parametrize("M,N,K,status", [
    (8192, 8192, (1 << 31) // (2 * 256), w.WS_ERR_INVALID_ARG),        # 256 K 2 bytes of an A panel reach 2^31
    (8192, 8192, (1 << 31) // (2 * 256) - 64, w.WS_OK),
    (8192, (1 << 31) // (4 * 256), 8192, w.WS_ERR_INVALID_ARG),        # 256 N 4 bytes of a C panel reach 2^31
    (8192, (1 << 31) // (4 * 256) - 128, 8192, w.WS_OK),
    ((1 << 30) + 1, 128, 64, w.WS_ERR_INVALID_ARG),                    # dimensions are capped at 2^30
    (1 << 30, 128, 64, w.WS_OK),
    (1 << 30, 1 << 20, 64, w.WS_ERR_INVALID_ARG),                      # 2^31 output tiles
])
def test_plan_size_limits(M, N, K, status):
    """The largest accepted problems: byte offsets inside one tile panel are
    32-bit, so T_M K 2, T_K N 2 and T_M N 4 must stay below 2^31."""
    s, info = w.ws_gemm_plan(M, N, K, cfg((256, 128, 64)), 256, 1)
    assert s == status, w.ws_gemm_status_str(s)
    if s == w.WS_OK:
        assert info.tiles == -(-M // 256) * -(-N // 128) and info.iters == -(-K // 64)
