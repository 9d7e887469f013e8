#!/usr/bin/env python
"""Benchmark of the warp-specialised GEMM on one MI355X.

Metric: bf16 GEMM TFLOP/s (and fraction of the dense MFMA peak) at
M = N = K = 8192, bf16 operands ~ N(0,1), fp32 output.  One step is one full
C = A B.  Operands are generated once (seeded, synthetic) and are resident in
HBM before the timed region starts.

    python bench.py [--gpus 1] [--steps 100] [--warmup 50] [--point TMxTNxTKxSxNPxNC[xSPLIT]]
                    [--workload NAME]

Prints one JSON line.  The default workload is the 8192^3 product above;
--workload runs another of the GEMM workloads (paper_2506_11209_amd/
workloads.py) at its own launch point, with the roofline taken against HBM
bandwidth when its arithmetic intensity is below the ridge point.  Also reported: the dominant kernel's roofline entry
(device time per launch from HIP events on the launch stream) and the CPU
oracle timed on this host's cores over a bounded sample of the same product.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "gemm_8192x8192x8192_bf16_normal"
# (TM, TN, TK, stages, producer waves, consumer waves, split): 256 x 256 tiles,
# eight consumer waves (two per SIMD) and four producer waves in one group (1:1)
DEFAULT_POINT = (256, 256, 64, 2, 4, 8, 1)
DEFAULT_LOAD_PATH = "registers"
PEAK_TFLOPS = 2500.0                      # MI355X dense bf16 / fp16 MFMA
PEAK_HBM_GBS = 8000.0                     # MI355X HBM3E
PEAK_CLOCK_MHZ = 2400.0                   # the clock the MFMA peak is quoted at
PROFILES = os.path.join(ROOT, "profiles")


def kernel_fingerprint(point=DEFAULT_POINT, dtype="bf16") -> str:
    """Hash of the machine code of the GEMM kernel that `point` launches, read
    from the built library (the counter records are tied to that code)."""
    from paper_2506_11209_amd.kernel_code import gemm_symbol, kernel_fingerprint as code_fingerprint
    from paper_2506_11209_amd.workloads import split_of, unpack
    tm, tn, tk, _stages, np_, nc, _ = unpack(point)
    return code_fingerprint(gemm_symbol(tm, tn, tk, nc, np_, split_of(point), bf16=(dtype == "bf16")))


def traffic_for(point_key: str, point=DEFAULT_POINT, dtype="bf16", workload=WORKLOAD):
    """HBM bytes per launch from the committed counter runs (profiles/
    *hbm_traffic*.json), if they were taken on this workload and launch point
    and on the machine code the library now holds for it; else None."""
    import glob
    fp = kernel_fingerprint(point, dtype)
    for path in sorted(glob.glob(os.path.join(PROFILES, "*hbm_traffic*.json"))):
        try:
            with open(path) as f:
                t = json.load(f)
        except (OSError, ValueError):
            continue
        if (t.get("kernel_fingerprint") == fp and t.get("point") == point_key
                and t.get("workload") == workload):
            return t.get("traffic_bytes_per_launch")
    return None


def copy_bandwidth(gib: float = 1.0, reps: int = 10) -> float:
    """Measured device copy bandwidth of this GPU in GB/s (read plus write
    bytes per second of a `gib` GiB tensor copy, HIP events around `reps`
    copies after a warm-up): the practical HBM reference beside the 8 TB/s
    peak for workloads below the ridge point."""
    import torch
    n = int(gib * (1 << 30)) // 2
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    for _ in range(reps):
        dst.copy_(src)
    ev[1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / reps
    del src, dst
    return 2.0 * 2 * n / (ms * 1e-3) / 1e9


def host_cpu() -> dict:
    """CPU model and thread counts of this host."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": usable, "logical_cpus": os.cpu_count()}


def _oracle_rate(wl, nthreads, target_s, lib):
    """TFLOP/s of the oracle on the first rows of wl's product (sized to take
    about target_s), with the number of rows and the seconds."""
    import numpy as np
    import oracle
    from paper_2506_11209_amd import inputs
    A, B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
    Ab, Bb = inputs.bits(A), inputs.bits(B)
    threads = nthreads or oracle.max_threads(lib)
    # size the sample from a probe of a few rows per thread (a probe of one
    # row per thread is dominated by thread start-up and undersizes it)
    cal_rows = min(wl.M, 4 * max(16 if nthreads != 1 else 2, threads))
    t0 = time.perf_counter()
    oracle.gemm_rows(Ab, Bb, wl.dtype, np.arange(cal_rows), nthreads=nthreads, lib=lib, with_abs=False)
    t_cal = time.perf_counter() - t0
    rows = int(max(1, min(wl.M, cal_rows * target_s / max(t_cal, 1e-3))))
    if rows >= 16:
        rows -= rows % 16
    t0 = time.perf_counter()
    oracle.gemm_rows(Ab, Bb, wl.dtype, np.arange(rows), nthreads=nthreads, lib=lib, with_abs=False)
    t = time.perf_counter() - t0
    return 2.0 * rows * wl.N * wl.K / t / 1e12, rows, t


def cpu_baseline(wl, target_s: float = 15.0):
    """The oracle (fp64 triple loop, as committed) on a sample of rows of C,
    on all host threads; plus single-thread timings of the 256^3 product
    (whole) and of a sample of the 4096^3 product."""
    import oracle
    from paper_2506_11209_amd.workloads import WORKLOADS
    lib = oracle.load()
    value, rows, t = _oracle_rate(wl, 0, target_s, lib)
    out = {"value": value, "unit": "TFLOP/s", "cores": oracle.max_threads(lib), "kind": "oracle",
           "sample": "%d of %d rows of C (%dx%d by %dx%d), including operand decode; %.1f s" % (
               rows, wl.M, wl.M, wl.K, wl.K, wl.N, t)}
    out.update(host_cpu())
    single = {}
    for name, tgt in (("gemm_256x256x256_f16_int4", 1.0), ("gemm_4096x4096x4096_bf16_normal", 6.0)):
        v, r, ts = _oracle_rate(WORKLOADS[name], 1, tgt, lib)
        single[name] = {"gflops": round(v * 1e3, 3), "rows": r, "seconds": round(ts, 3)}
    out["single_thread"] = single
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--point", default=None, help="TMxTNxTKxSTAGESxNPxNC[xSPLIT]")
    ap.add_argument("--load-path", default=DEFAULT_LOAD_PATH, choices=("registers", "dma"))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--cold-flush-mib", type=int, default=0,
                    help="write a buffer of this many MiB before every timed launch (outside its events), "
                         "so each launch starts with its operands out of the caches; the roofline entry "
                         "then comes from the launch events alone")
    ap.add_argument("--min-warmup-s", type=float, default=0.5,
                    help="warm up for at least this long, and until two batches of 10 agree within 1%%")
    a = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the GEMM library has no multi-GPU path "
              "(requested --gpus %d, WORLD_SIZE %d)" % (a.gpus, world), file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_11209_amd import inputs
    from paper_2506_11209_amd import wsgemm as w
    from paper_2506_11209_amd.timing import summary, time_launches
    from paper_2506_11209_amd.workloads import WORKLOADS, parse_point, point_key, split_of, unpack

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if a.workload not in WORKLOADS:
        print("unknown workload %s; one of %s" % (a.workload, sorted(WORKLOADS)), file=sys.stderr)
        sys.exit(2)
    wl = WORKLOADS[a.workload]
    if a.point:
        point = parse_point(a.point)
    else:
        point = DEFAULT_POINT if wl.name == WORKLOAD else wl.points[0]
    tm, tn, tk, stages, np_, nc, split = unpack(point)
    A, B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
    Ad, Bd = A.cuda(), B.cuda()
    del A, B
    C = torch.empty((wl.M, wl.N), dtype=torch.float32, device="cuda")
    g = w.WsGemm(wl.M, wl.N, wl.K, (tm, tn, tk), stages, np_, nc, wl.dtype, a.load_path, split=split)
    stream = torch.cuda.current_stream()
    a_p, b_p, c_p, s_p = Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(), stream.cuda_stream

    def step():
        g.run_ptrs(a_p, b_p, c_p, s_p)

    # warm up by count and by time (the clock ramps over the first launches);
    # the launch clock accumulators are cleared just before the timed region
    flush = None
    if a.cold_flush_mib > 0:
        junk = torch.empty(a.cold_flush_mib << 18, dtype=torch.float32, device="cuda")

        def flush():
            junk.fill_(1.0)
    dev, wall_ms, wu = time_launches(step, a.steps, a.warmup, min_warmup_s=a.min_warmup_s,
                                     with_warmup=True, before_timed=lambda: g.clock_mhz(stream),
                                     between=flush)
    clock_mhz, clock_n = g.clock_mhz(stream)
    st = g.sync_status(stream)
    if st != w.WS_OK:
        print("kernel reported %s" % w.ws_gemm_status_str(st), file=sys.stderr)
        sys.exit(1)
    sm = summary(dev)
    value = wl.flops / (wall_ms * 1e-3) / 1e12
    pkey = point_key(point) + "/" + a.load_path
    # roofline of the kernel: MFMA peak, or HBM bandwidth below the ridge point
    if wl.flops / wl.bytes >= PEAK_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        bound, unit, peak = "mfma", "TFLOP/s", PEAK_TFLOPS
        achieved = wl.flops / (sm["mean_ms"] * 1e-3) / 1e12
    else:
        bound, unit, peak = "hbm", "GB/s", PEAK_HBM_GBS
        achieved = wl.bytes / (sm["mean_ms"] * 1e-3) / 1e9
    if wl.name == WORKLOAD:
        metric = "bf16 GEMM TFLOP/s at 8192^3 (fraction of dense MFMA peak in pct_mfma_peak)"
    else:
        metric = "%s GEMM TFLOP/s at %dx%dx%d" % (wl.dtype, wl.M, wl.N, wl.K)
    out = {
        "metric": metric,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(wall_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "pct_mfma_peak": round(100.0 * value / PEAK_TFLOPS, 2),
        "config": {"workload": wl.name, "M": wl.M, "N": wl.N, "K": wl.K,
                   "tile": [tm, tn, tk], "stages": stages, "producer_waves": np_,
                   "consumer_waves": nc, "split": "%d:1" % split_of(point),
                   "load_path": a.load_path, "grid": g.info.grid, "rounds": g.info.rounds},
        "roofline": {"bound": bound, "achieved": round(achieved, 2), "peak": peak,
                     "unit": unit, "frac": round(achieved / peak, 4),
                     "traffic": traffic_for(pkey, point, wl.dtype, wl.name) if np_ > 0 else None,
                     "kernel": ("ws_gemm_kernel<%d,%d,%d,%d,%d,%d,%s>" % (tm, tn, tk, nc, np_, split_of(point),
                                                                          wl.dtype)
                                if np_ > 0 else "ws_sync_kernel<%d,%d,%d,%d,%s>" % (tm, tn, tk, nc, wl.dtype)),
                     "algorithmic_bytes": wl.bytes, "flop": wl.flops,
                     "achieved_at_median": round(achieved * sm["mean_ms"] / sm["median_ms"], 2),
                     "launch_ms": {k: round(v, 5) if isinstance(v, float) else v for k, v in sm.items()},
                     "clock_mhz": round(clock_mhz, 1) if clock_mhz else None,
                     "clock_launches": clock_n,
                     "frac_at_clock": (round(achieved / (peak * clock_mhz / PEAK_CLOCK_MHZ), 4)
                                       if clock_mhz and bound == "mfma" else None)},
        "warmup_record": wu,
    }
    if a.cold_flush_mib > 0:
        out["cold_flush_mib"] = a.cold_flush_mib  # value includes the flushes; roofline does not
    g.close()
    if bound == "hbm":
        # against what this machine's HBM sustains in practice, measured after the timed region
        cbw = copy_bandwidth()
        out["roofline"]["copy_gbs"] = round(cbw, 1)
        out["roofline"]["frac_of_copy"] = round(achieved / cbw, 4)
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
