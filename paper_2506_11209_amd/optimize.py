"""Pick a launch configuration with the performance model (paper, Section 3.2,
"Finding optimal solutions"), by exhaustive search over the compiled
configurations instead of an SMT solver.

    python -m paper_2506_11209_amd.optimize --calib calib.json --mnk 8192,8192,8192 \
        [--objective time|wait] [--top 10] [--measure] [--out ranking.jsonl]

Every launchable (tile, stages, producer/consumer waves) of the problem is
predicted with the calibrated model (library ws_model_predict, persistent
schedule); the list is ranked by predicted time (first objective) or by the
predicted total MATH wait (second objective).  With --measure every candidate
is also timed on the GPU, and the report gives the measured time of the
predicted best, the measured best, the regret and the rank correlation
between predicted and measured times.
"""
from __future__ import annotations

import argparse
import json
import statistics
import sys
import time

from paper_2506_11209_amd.model import candidates, load_calibration, load_cost_table, optimize


def spearman(xs, ys):
    def ranks(v):
        order = sorted(range(len(v)), key=lambda i: v[i])
        r = [0.0] * len(v)
        for k, i in enumerate(order):
            r[i] = float(k)
        return r
    rx, ry = ranks(xs), ranks(ys)
    mx, my = statistics.fmean(rx), statistics.fmean(ry)
    num = sum((a - mx) * (b - my) for a, b in zip(rx, ry))
    den = (sum((a - mx) ** 2 for a in rx) * sum((b - my) ** 2 for b in ry)) ** 0.5
    return num / den if den else float("nan")


def measure(rows, M, N, K, load_path, steps, warmup):
    """Time every candidate on the GPU: two passes, the second in reverse
    order, after a warm-up of the clock; each candidate keeps the lower of its
    two medians, so that no candidate is timed only at a pass's cold start."""
    import torch

    from paper_2506_11209_amd import wsgemm as w
    from paper_2506_11209_amd.timing import time_launches
    torch.manual_seed(0)
    A = torch.randn(M, K, device="cuda").to(torch.bfloat16)
    B = torch.randn(K, N, device="cuda").to(torch.bfloat16)
    C = torch.empty(M, N, device="cuda")
    st = torch.cuda.current_stream().cuda_stream

    def median_us(r, nsteps, nwarm, min_seconds=0.0):
        g = w.WsGemm(M, N, K, r["tile"], r["stages"], r["producer_waves"], r["consumer_waves"], "bf16",
                     load_path, split=r["split"])
        try:
            t0 = time.perf_counter()
            while True:
                dev, _ = time_launches(lambda: g.run_ptrs(A.data_ptr(), B.data_ptr(), C.data_ptr(), st),
                                       nsteps, nwarm)
                if time.perf_counter() - t0 >= min_seconds:
                    return statistics.median(dev) * 1e3
        finally:
            g.close()

    if rows:
        median_us(rows[0], steps, 0, min_seconds=0.5)  # bring the clock up before the first candidate
    for r in rows:
        r["measured_pass_us"] = [median_us(r, steps, warmup)]
    for r in reversed(rows):
        r["measured_pass_us"].append(median_us(r, steps, warmup))
        r["measured_us"] = min(r["measured_pass_us"])
    for r in rows:
        print("%-14s P=%d %d:%d/%d  predicted %9.1f us  measured %9.1f us" % (
            "x".join(map(str, r["tile"])), r["stages"], r["producer_waves"], r["consumer_waves"], r["split"],
            r["time_us"], r["measured_us"]), file=sys.stderr, flush=True)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--calib", required=True)
    ap.add_argument("--mnk", default="8192,8192,8192")
    ap.add_argument("--objective", default="time", choices=("time", "wait"))
    ap.add_argument("--load-path", default="registers")
    ap.add_argument("--num-cus", type=int, default=256)
    ap.add_argument("--top", type=int, default=10)
    ap.add_argument("--costs", default="fit", choices=("fit", "table"),
                    help="fit: linear costs of Section 4.2; table: measured per-tile costs where available")
    ap.add_argument("--measure", action="store_true")
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    M, N, K = (int(x) for x in a.mnk.split(","))
    cal = load_calibration(a.calib)
    params = {s: cal[(s, a.load_path)] for s in (1, 2) if (s, a.load_path) in cal}
    cands = [c for c in candidates(M, N, K, num_cus=a.num_cus, load_path=a.load_path) if c[5] in params]
    table = load_cost_table(a.calib) if a.costs == "table" else None
    rows = optimize(M, N, K, params, cands, a.objective, table=table, load_path=a.load_path)
    for i, r in enumerate(rows):
        r["predicted_rank"] = i
    report = {"M": M, "N": N, "K": K, "objective": a.objective, "costs": a.costs, "candidates": len(rows),
              "predicted_best": rows[0] if rows else None}
    if a.measure and rows:
        measure(rows, M, N, K, a.load_path, a.steps, a.warmup)
        best = min(rows, key=lambda r: r["measured_us"])
        report["measured_best"] = best
        report["regret"] = rows[0]["measured_us"] / best["measured_us"] - 1.0
        report["spearman_time"] = spearman([r["time_us"] for r in rows], [r["measured_us"] for r in rows])
        report["top1_hit"] = rows[0] is best
    if a.out:
        with open(a.out, "w") as f:
            for r in rows:
                f.write(json.dumps(r) + "\n")
    for r in rows[:a.top]:
        print("%-14s P=%d %d:%d/%d slots=%d predicted %9.1f us wait %9.1f us%s" % (
            "x".join(map(str, r["tile"])), r["stages"], r["producer_waves"], r["consumer_waves"], r["split"],
            r["slots"], r["time_us"], r["wait_us"],
            ("  measured %9.1f us" % r["measured_us"]) if "measured_us" in r else ""), file=sys.stderr)
    print(json.dumps(report, default=str))


if __name__ == "__main__":
    main()
