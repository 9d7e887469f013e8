"""Prediction accuracy of the performance model on this GPU (paper, Section 4.2,
"Estimate the Execution Time of the GeMM-WS Kernel").

    python -m paper_2506_11209_amd.model_eval --calib calib.json [--grid accuracy|bench] [--out eval.jsonl]

Times the GEMM kernel on a grid of problem sizes and launch configurations,
predicts each time with the calibrated model (library ``ws_model_predict``)
and reports the relative error |predicted - measured| / measured: its mean
and maximum over the grid, the paper's two accuracy figures.  Two readings of
the schedule are evaluated side by side: the per-round pipeline the paper
prints (Section 2.1/2.2) and the persistent grid the kernel runs.

Grids:
  accuracy  M, N in {2048, 4096, 8192}, K in {1024, 4096, 8192}, tiles
            {128x128x64, 256x128x64, 128x256x64, 64x64x64, 128x128x32,
            128x256x32}, 3 stages (2 where 3 do not fit), one and two DMA
            wave groups;
  bench     the 8192^3 launch points of the sweep;
  paper     the paper's own evaluation grid (Section 4.2): M, N, K every
            multiple of 128 up to 1024, tiles (64|128) x (64|128) x 64,
            3 stages, one and two DMA wave groups.
With --costs table, tiles without measured costs use the linear fit.  With
--fixed launch, T_INIT and T_EPILOGUE are measured for every launch point
(the empty and epilogue-only calibration kernels with that point's own
launch) instead of once, on the calibration file's launch.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import statistics
import sys

import torch

from paper_2506_11209_amd import wsgemm as w
from paper_2506_11209_amd.model import load_calibration, load_cost_table, predict, predict_costs
from paper_2506_11209_amd.timing import time_launches
from paper_2506_11209_amd.workloads import WORKLOADS, split_of, unpack

LDS_LIMIT = 163840


def fits(tile, stages):
    tm, tn, tk = tile
    return 256 + stages * 2 * (tm * tk + tk * tn) <= LDS_LIMIT


def accuracy_grid():
    tiles = ((128, 128, 64), (256, 128, 64), (128, 256, 64), (64, 64, 64), (128, 128, 32),
             (128, 256, 32))
    out = []
    for M in (2048, 4096, 8192):
        for N in (2048, 4096, 8192):
            for K in (1024, 4096, 8192):
                for tile in tiles:
                    P = 3 if fits(tile, 3) else 2
                    for split in (1, 2):
                        out.append((M, N, K, tile, P, split))
    return out


def bench_grid():
    wl = WORKLOADS["gemm_8192x8192x8192_bf16_normal"]
    out = []
    for pt in wl.points:
        tm, tn, tk, P, np_, nc, _ = unpack(pt)
        # the synchronous kernel's points have no producers; the model is
        # calibrated for split groups of four producer waves
        if np_ > 0 and np_ == nc * split_of(pt) and nc == 4 and fits((tm, tn, tk), P):
            out.append((wl.M, wl.N, wl.K, (tm, tn, tk), P, split_of(pt)))
    return out


def paper_grid():
    sizes = range(128, 1025, 128)
    tiles = ((64, 64, 64), (64, 128, 64), (128, 64, 64), (128, 128, 64))
    return [(M, N, K, tile, 3, split) for M in sizes for N in sizes for K in sizes for tile in tiles
            for split in (1, 2)]


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--calib", required=True)
    ap.add_argument("--grid", default="accuracy", choices=("accuracy", "bench", "paper"))
    ap.add_argument("--quiet", action="store_true", help="no per-launch line on stderr")
    ap.add_argument("--fixed", default="file", choices=("file", "launch"),
                    help="T_INIT / T_EPILOGUE from the calibration file, or measured per launch point")
    ap.add_argument("--load-path", default="registers")
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--costs", default="fit", choices=("fit", "table"),
                    help="fit: the linear cost model of Section 4.2; table: costs measured per tile")
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    cal = load_calibration(a.calib)
    table = load_cost_table(a.calib) if a.costs == "table" else None
    grid = {"accuracy": accuracy_grid, "bench": bench_grid, "paper": paper_grid}[a.grid]()
    Mx = max(g[0] for g in grid)
    Nx = max(g[1] for g in grid)
    Kx = max(g[2] for g in grid)
    torch.manual_seed(0)
    A = torch.randn(Mx, Kx, device="cuda").to(torch.bfloat16)
    B = torch.randn(Kx, Nx, device="cuda").to(torch.bfloat16)
    C = torch.empty(Mx, Nx, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    rows = []
    fout = open(a.out, "w") if a.out else None
    for (M, N, K, tile, P, split) in grid:
        g = w.WsGemm(M, N, K, tile, P, 4 * split, 4, "bf16", a.load_path)
        try:
            ap_, bp, cp = A.data_ptr(), B.data_ptr(), C.data_ptr()
            dev, _ = time_launches(lambda: g.run_ptrs(ap_, bp, cp, st), a.steps, a.warmup)
            meas = statistics.median(dev) * 1e3
            slots = g.info.grid
        finally:
            g.close()
        params = cal[(split, a.load_path)]
        if a.fixed == "launch":
            fixed = {}
            for kind in ("empty", "epilogue"):
                gk = w.WsGemm(M, N, K, tile, P, 4 * split, 4, "bf16", a.load_path, calibration=kind)
                try:
                    dev, _ = time_launches(lambda: gk.run_ptrs(ap_, bp, cp, st), a.steps, a.warmup)
                    fixed[kind] = statistics.median(dev) * 1e3
                    rounds = gk.info.rounds
                finally:
                    gk.close()
            params = dataclasses.replace(params, t_init=fixed["empty"],
                                         t_epilogue=max(fixed["epilogue"] - fixed["empty"], 0.0) / rounds)
        rec = {"M": M, "N": N, "K": K, "tile": tile, "stages": P, "split": split,
               "load_path": a.load_path, "measured_us": meas, "slots": slots}
        for name, persistent in (("per_round", False), ("persistent", True)):
            costs = table.get((split, a.load_path, tuple(tile))) if table is not None else None
            if costs is not None:
                t_math, t_la, t_lb = costs
                pr = predict_costs(M, N, K, tile, P, slots, params, t_math, t_la, t_lb,
                                   two_dma=(split == 2), persistent=persistent)
            else:
                pr = predict(M, N, K, tile, P, slots, params, two_dma=(split == 2),
                             persistent=persistent)
            rec[name + "_us"] = pr["total_us"]
            rec[name + "_err"] = (pr["total_us"] - meas) / meas
            rec["rounds"], rec["iters"] = pr["rounds"], pr["iters"]
            rec["t_math"], rec["t_load_a"], rec["t_load_b"] = pr["t_math"], pr["t_load_a"], pr["t_load_b"]
        rec["costs"] = "table" if costs is not None else "fit"
        rec["t_init_us"], rec["t_epilogue_us"] = params.t_init, params.t_epilogue
        rows.append(rec)
        if fout:
            fout.write(json.dumps(rec) + "\n")
            fout.flush()
        if not a.quiet or len(rows) % 256 == 0:
            print("%5d %5d %5d %-15s P=%d %d:1  measured %9.1f us  per-round %9.1f (%+6.1f%%)  persistent %9.1f (%+6.1f%%)" % (
                M, N, K, "x".join(map(str, tile)), P, split, meas, rec["per_round_us"],
                100 * rec["per_round_err"], rec["persistent_us"], 100 * rec["persistent_err"]),
                file=sys.stderr, flush=True)
    summary = {"points": len(rows), "grid": a.grid, "load_path": a.load_path, "costs": a.costs,
               "fixed": a.fixed}
    for name in ("per_round", "persistent"):
        errs = [abs(r[name + "_err"]) for r in rows]
        summary[name] = {"mean_abs_err": statistics.fmean(errs), "max_abs_err": max(errs)}
    print(json.dumps(summary))
    if fout:
        fout.write(json.dumps({"summary": summary}) + "\n")
        fout.close()


if __name__ == "__main__":
    main()
