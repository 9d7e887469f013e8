"""Sweep launcher: time the warp-specialised GEMM over tile tuples, stage
depths and producer/consumer wave splits on one GPU.

    python -m paper_2506_11209_amd.sweep --workload gemm_8192x8192x8192_bf16_normal \
        [--steps 30] [--warmup 5] [--out sweep.jsonl]

One JSON line per launch point: device time (mean/median/std over HIP-event
pairs), TFLOP/s, fraction of the dense MFMA peak and of the HBM roofline, and
the largest error on 16 sampled rows of C against a float32 torch product,
scaled by |A||B| (a sanity figure; the parity tests check against the CPU
oracle).
Points whose ring does not fit in LDS are reported with their status.
Appends to --out and skips points already present there, so an interrupted
sweep resumes.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import torch

from paper_2506_11209_amd import inputs
from paper_2506_11209_amd import wsgemm as w
from paper_2506_11209_amd.timing import summary, time_launches
from paper_2506_11209_amd.workloads import WORKLOADS, parse_point, point_key, split_of, unpack

PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0}  # MI355X dense MFMA
PEAK_HBM_GBS = 8000.0


def measure_point(wl, point, Ad, Bd, C, steps, warmup, load_path="registers", min_warmup_s=0.3):
    tm, tn, tk, stages, np_, nc, split = unpack(point)
    cfg = w.config((tm, tn, tk), stages, np_, nc, wl.dtype, load_path, split)
    s, h = w.ws_gemm_create(wl.M, wl.N, wl.K, cfg)
    rec = {"workload": wl.name, "tile": [tm, tn, tk], "stages": stages, "producer_waves": np_,
           "consumer_waves": nc, "split": "%d:1" % split_of(point), "load_path": load_path,
           "point": point_key(point) + "/" + load_path}
    if s != w.WS_OK:
        rec["status"] = w.ws_gemm_status_str(s)
        return rec
    try:
        _, info = w.ws_gemm_query(h)
        stream = torch.cuda.current_stream().cuda_stream
        a, b, c = Ad.data_ptr(), Bd.data_ptr(), C.data_ptr()

        def launch():
            st = w.ws_gemm_run(h, a, b, c, stream)
            if st != w.WS_OK:
                raise RuntimeError(w.ws_gemm_status_str(st))

        dev, wall = time_launches(launch, steps, warmup, min_warmup_s=min_warmup_s,
                                  before_timed=lambda: w.ws_gemm_clock(h, stream))
        _, cyc, ticks, nclk = w.ws_gemm_clock(h, stream)
        rec["clock_mhz"] = 100.0 * cyc / ticks if ticks else None
        st = w.ws_gemm_sync_status(h, stream)
        if st != w.WS_OK:
            rec["status"] = w.ws_gemm_status_str(st)
            return rec
    finally:
        w.ws_gemm_destroy(h)
    sm = summary(dev)
    t = sm["mean_ms"] * 1e-3
    tflops = wl.flops / t / 1e12
    rows = torch.linspace(0, wl.M - 1, 16, device=Ad.device).long()
    Ar, Bf = Ad[rows].float(), Bd.float()
    scale = (Ar.abs() @ Bf.abs()).clamp_min(torch.finfo(torch.float32).tiny)
    max_scaled_err = float(((C[rows] - Ar @ Bf).abs() / scale).max())
    del Bf
    rec.update({
        "status": "ok", "plan": info.as_dict(), "device_ms": sm, "wall_ms_per_launch": wall,
        "tflops": tflops, "frac_mfma_peak": tflops / PEAK_TFLOPS[wl.dtype],
        "frac_mfma_peak_at_clock": (tflops / (PEAK_TFLOPS[wl.dtype] * rec["clock_mhz"] / 2400.0)
                                    if rec.get("clock_mhz") else None),
        "hbm_gbs_algorithmic": wl.bytes / t / 1e9, "frac_hbm_roofline": wl.bytes / t / 1e9 / PEAK_HBM_GBS,
        "max_scaled_err": max_scaled_err,
    })
    return rec


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="gemm_8192x8192x8192_bf16_normal", choices=sorted(WORKLOADS))
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--out", default=None)
    ap.add_argument("--load-paths", default="registers,dma",
                    help="comma-separated producer load paths to sweep (registers, dma)")
    ap.add_argument("--points", default=None,
                    help="comma-separated TMxTNxTKxSTAGESxNPxNC[xSPLIT] list (default: the workload's)")
    ap.add_argument("--min-warmup-s", type=float, default=0.3,
                    help="warm each point up for at least this long (0: exactly --warmup launches, "
                         "as counter runs need)")
    a = ap.parse_args(argv)
    wl = WORKLOADS[a.workload]
    points = wl.points
    if a.points:
        points = tuple(parse_point(p) for p in a.points.split(","))
    done = set()
    if a.out and os.path.exists(a.out):
        for line in open(a.out):
            try:
                r = json.loads(line)
                if r.get("workload") == wl.name and r.get("status") == "ok":
                    done.add(r["point"])
            except ValueError:
                pass
    A, B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
    Ad, Bd = A.cuda(), B.cuda()
    C = torch.empty((wl.M, wl.N), dtype=torch.float32, device="cuda")
    del A, B
    for p in points:
        for lp in a.load_paths.split(","):
            key = point_key(p) + "/" + lp
            if key in done:
                continue
            print("sweep point %s" % key, file=sys.stderr, flush=True)
            rec = measure_point(wl, p, Ad, Bd, C, a.steps, a.warmup, lp, a.min_warmup_s)
            line = json.dumps(rec)
            print(line, flush=True)
            if a.out:
                with open(a.out, "a") as f:
                    f.write(line + "\n")


if __name__ == "__main__":
    main()
