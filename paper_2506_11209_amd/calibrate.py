"""Calibrate the performance model on this GPU (paper, Section 4.2).

    python -m paper_2506_11209_amd.calibrate [--load-paths registers,dma] [--out calib.json]

For each producer arrangement (one DMA wave group loading A then B, and two
loading A and B concurrently) and load path, with the calibration kernels of
the library (``ws_gemm_create_calibration``) on the launch of an 8192 x 8192
output (full grid, several rounds; --mn sets another square output):

  T_INIT      the empty kernel's time;
  T_EPILOGUE  (epilogue-only kernel time - T_INIT) / rounds, at least 0
              (at a one-round launch the difference is a fraction of a
              microsecond, so both kernels take FIXED_LAUNCHES timed
              launches);
  T_LOAD-A    load-only time per K-iteration of one workgroup, for two A-tile
              sizes, from the difference of two K so that launch, fill and
              drain cancel;
  T_MATH      math-only time per K-iteration for the same two tiles.

The two tiles of a pair run the same consumer code (128x128x64 with
256x128x64 for one DMA group; 128x128x64 with 128x128x32 for two, whose
largest tiles take another consumer variant).  The two-point fits of Section
4.2 turn the pairs into throughput and startup latency.  T_LOAD-B is
measured too and reported against the fitted line (the model assumes A and
B loads cost the same per element).

With --table, T_MATH, T_LOAD-A, T_LOAD-B and the time of loading both tiles
(the producers' own rate, WS_CALIB_LOAD_AB) are also measured directly for
every tile of the accuracy grid (model_eval.py), so that the event model can
be evaluated apart from the linear cost model; --table-tiles paper measures
the tiles of the paper's own grid instead.  The accuracy table also holds
the eight-consumer 256 x 256 launches (four producer waves in `split`
groups), whose consumer the linear fits do not describe: the optimizer ranks
them with these measured costs only.  Writes one JSON document with every
raw measurement.
"""
from __future__ import annotations

import argparse
import json
import statistics
import sys
import time

import torch

from paper_2506_11209_amd import wsgemm as w
from paper_2506_11209_amd.model import Params, params_dict, two_point_fit
from paper_2506_11209_amd.timing import time_launches

MN = 8192
K_PAIR = (1024, 4096)
PAIRS = {1: ((128, 128, 64), (256, 128, 64)), 2: ((128, 128, 64), (128, 128, 32))}
TABLE_TILES = {
    "accuracy": ((128, 128, 64), (256, 128, 64), (128, 256, 64), (64, 64, 64), (128, 128, 32),
                 (128, 256, 32)),
    "paper": ((64, 64, 64), (64, 128, 64), (128, 64, 64), (128, 128, 64)),
}
# eight consumer waves, four producer waves: (tile, stages) measured with the accuracy table
EIGHT_CONSUMER_TILES = (((256, 256, 64), 2), ((256, 256, 32), 4))
LDS_LIMIT = 163840
FIXED_LAUNCHES = 200


def stages_for(tile):
    tm, tn, tk = tile
    return 3 if 256 + 3 * 2 * (tm * tk + tk * tn) <= LDS_LIMIT else 2


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_us(kind, M, N, K, tile, np_, load_path, A, B, C, steps, warmup, nc=4, split=0, stages=None):
    g = w.WsGemm(M, N, K, tile, stages or stages_for(tile), np_, nc, "bf16", load_path, calibration=kind,
                 split=split)
    try:
        st = torch.cuda.current_stream().cuda_stream
        a, b, c = A.data_ptr(), B.data_ptr(), C.data_ptr()
        dev, _ = time_launches(lambda: g.run_ptrs(a, b, c, st), steps, warmup)
        s = g.sync_status()
        if s != w.WS_OK:
            raise RuntimeError("%s: %s" % (kind, w.ws_gemm_status_str(s)))
        return statistics.median(dev) * 1e3, g.info.rounds
    finally:
        g.close()


def fixed_costs_us(M, tile, np_, load_path, A, B, C, warmup, nc=4, split=0, stages=None):
    """Empty-kernel and epilogue-only-kernel times (us) of one launch point
    (medians of FIXED_LAUNCHES launches each) and the launch's rounds."""
    P = stages or stages_for(tile)
    empty = w.WsGemm(M, M, tile[2], tile, P, np_, nc, "bf16", load_path, calibration="empty", split=split)
    epi = w.WsGemm(M, M, tile[2], tile, P, np_, nc, "bf16", load_path, calibration="epilogue", split=split)
    try:
        st = torch.cuda.current_stream().cuda_stream
        a, b, c = A.data_ptr(), B.data_ptr(), C.data_ptr()
        samples = {}
        for kind, g in (("empty", empty), ("epilogue", epi)):
            samples[kind], _ = time_launches(lambda: g.run_ptrs(a, b, c, st), FIXED_LAUNCHES, warmup)
        for g in (empty, epi):
            s = g.sync_status()
            if s != w.WS_OK:
                raise RuntimeError("fixed costs: %s" % w.ws_gemm_status_str(s))
        return (statistics.median(samples["empty"]) * 1e3, statistics.median(samples["epilogue"]) * 1e3,
                epi.info.rounds)
    finally:
        empty.close()
        epi.close()


def per_iteration_us(kind, tile, np_, load_path, bufs, steps, warmup, nc=4, split=0, stages=None):
    """Time one workgroup spends per K-iteration, from two values of K."""
    A, B, C = bufs
    mn = C.shape[0]
    tk = tile[2]
    t1, W = kernel_us(kind, mn, mn, K_PAIR[0], tile, np_, load_path, A, B, C, steps, warmup, nc, split, stages)
    t2, _ = kernel_us(kind, mn, mn, K_PAIR[1], tile, np_, load_path, A, B, C, steps, warmup, nc, split, stages)
    iters = W * (K_PAIR[1] - K_PAIR[0]) // tk
    return (t2 - t1) / iters, {"t_k1_us": t1, "t_k2_us": t2, "rounds": W}


def costs(tile, np_, load_path, bufs, steps, warmup, nc=4, split=0, stages=None):
    """Measured per-K-iteration T_LOAD-A, T_LOAD-B and T_MATH of one tile."""
    kw = dict(nc=nc, split=split, stages=stages)
    la, ra = per_iteration_us("load_a", tile, np_, load_path, bufs, steps, warmup, **kw)
    lb, rb = per_iteration_us("load_b", tile, np_, load_path, bufs, steps, warmup, **kw)
    mm, rm = per_iteration_us("math", tile, np_, load_path, bufs, steps, warmup, **kw)
    return (la, ra), (lb, rb), (mm, rm)


def calibrate(split, load_path, bufs, steps, warmup, table, eight=()):
    """table: None, or the tiles to measure one by one; eight: (tile, stages)
    of eight-consumer launches to add to the table."""
    np_ = 4 * split
    A, B, C = bufs
    mn = C.shape[0]
    tile0 = PAIRS[split][0]
    t_init, t_epi_kernel, W = fixed_costs_us(mn, tile0, np_, load_path, A, B, C, warmup)
    t_epi = max(t_epi_kernel - t_init, 0.0) / W  # a difference within the noise can come out below 0
    raw = {"t_init_us": t_init, "epilogue_kernel_us": t_epi_kernel, "epilogue_rounds": W,
           "fixed_cost_launches": FIXED_LAUNCHES}
    loads, loads_b, maths = [], [], []
    for tile in PAIRS[split]:
        tm, tn, tk = tile
        (la, ra), (lb, rb), (mm, rm) = costs(tile, np_, load_path, bufs, steps, warmup)
        loads.append({"tile": tile, "elements": tm * tk, "t_us": la, **ra})
        loads_b.append({"tile": tile, "elements": tk * tn, "t_us": lb, **rb})
        maths.append({"tile": tile, "macs": tm * tn * tk, "t_us": mm, **rm})
        log("split %d %s tile %s: load A %.4f us, load B %.4f us, math %.4f us per K-iteration" % (
            split, load_path, tile, la, lb, mm))
    lt, ll = two_point_fit(loads[0]["elements"], loads[0]["t_us"], loads[1]["elements"], loads[1]["t_us"])
    ct, cl = two_point_fit(maths[0]["macs"], maths[0]["t_us"], maths[1]["macs"], maths[1]["t_us"])
    for rec in loads_b:
        rec["fit_us"] = rec["elements"] / lt + ll
    p = Params(t_init, t_epi, ct, cl, lt, ll)
    rec = {"split": split, "load_path": load_path, "params": params_dict(p), "raw": raw,
           "load_a": loads, "load_b": loads_b, "math": maths}
    if table:
        rows = []
        for tile in table:
            (la, _), (lb, _), (mm, _) = costs(tile, np_, load_path, bufs, steps, warmup)
            lab, _ = per_iteration_us("load_ab", tile, np_, load_path, bufs, steps, warmup)
            rows.append({"tile": tile, "stages": stages_for(tile), "t_load_a": la, "t_load_b": lb,
                         "t_load_ab": lab, "t_math": mm})
            log("table split %d %s tile %s: load A %.4f  load B %.4f  load A+B %.4f  math %.4f us" % (
                split, load_path, tile, la, lb, lab, mm))
        for tile, P in eight:
            kw = dict(nc=8, split=split, stages=P)
            (la, _), (lb, _), (mm, _) = costs(tile, 4, load_path, bufs, steps, warmup, **kw)
            lab, _ = per_iteration_us("load_ab", tile, 4, load_path, bufs, steps, warmup, **kw)
            rows.append({"tile": tile, "stages": P, "consumer_waves": 8, "producer_waves": 4, "t_load_a": la,
                         "t_load_b": lb, "t_load_ab": lab, "t_math": mm})
            log("table split %d %s tile %s, 8 + 4 waves: load A %.4f  load B %.4f  load A+B %.4f  math %.4f us"
                % (split, load_path, tile, la, lb, lab, mm))
        rec["table"] = rows
    return rec


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--load-paths", default="registers")
    ap.add_argument("--splits", default="1,2")
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--table", action="store_true", help="also measure every tile of the evaluation grid")
    ap.add_argument("--table-tiles", default="accuracy", choices=tuple(TABLE_TILES))
    ap.add_argument("--mn", type=int, default=MN, help="rows and columns of the calibration output")
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    torch.manual_seed(0)
    mn = a.mn
    A = torch.randn(mn, K_PAIR[1], device="cuda").to(torch.bfloat16)
    B = torch.randn(K_PAIR[1], mn, device="cuda").to(torch.bfloat16)
    C = torch.empty(mn, mn, device="cuda")
    bufs = (A, B, C)
    # warm the clock up before the first measurement
    g = w.WsGemm(mn, mn, K_PAIR[1], (256, 128, 64), 3, 4, 4, "bf16")
    time_launches(lambda: g(A, B, C), 1, 50)
    g.close()
    out = {"device": torch.cuda.get_device_name(0), "time": time.strftime("%Y-%m-%d %H:%M:%S"),
           "problem": {"M": mn, "N": mn, "K_pair": K_PAIR, "pairs": {str(k): v for k, v in PAIRS.items()}},
           "calibrations": []}
    for lp in a.load_paths.split(","):
        for split in (int(x) for x in a.splits.split(",")):
            eight = EIGHT_CONSUMER_TILES if a.table and a.table_tiles == "accuracy" else ()
            rec = calibrate(split, lp, bufs, a.steps, a.warmup, TABLE_TILES[a.table_tiles] if a.table else None,
                            eight)
            out["calibrations"].append(rec)
            log("split %d %s: %s" % (split, lp, json.dumps(rec["params"])))
    text = json.dumps(out, indent=1)
    if a.out:
        with open(a.out, "w") as f:
            f.write(text + "\n")
    print(text)


if __name__ == "__main__":
    main()
