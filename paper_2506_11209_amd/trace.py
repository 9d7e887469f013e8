"""Event traces of the warp-specialised GEMM (the events of the paper's
Section 2.2, measured on the GPU).

    python -m paper_2506_11209_amd.trace [--workload NAME] [--point TMxTNxTKxSxNPxNC[xSPLIT]] [--wgs 4]
        [--warmup 20]

For each traced workgroup and K-iteration q the kernel stamps (shader clock):
issue of the A and B tiles (S_a, S_b), their landing in LDS, the consumer
observing the slot full, the consumer's MFMA start (S_m) and the slot
release.  This module runs one traced launch and reduces the stamps to the
quantities the model uses: load time per K-iteration, MATH time per
K-iteration, consumer waiting time (Wait(i) of Section 3.2) and epilogue time.
The stamps count shader clocks; the traced launch is timed with HIP events,
so the clock during it (stamped span / duration) converts them to us.
"""
from __future__ import annotations

import argparse
import json

import numpy as np

EVENTS = ("issue_a", "issue_b", "land_a", "land_b", "ready", "mma_start", "release", "epilogue_end")


def run_traced(wl, point, wgs=4, Ad=None, Bd=None, load_path="registers", warmup=0, pairs=1):
    """`pairs` untraced and traced launches, alternating, after `warmup`
    untraced ones; returns (records [wgs, iters, 8] uint32 of the last traced
    launch, plan dict with the median durations in us of the traced and the
    untraced launches under "traced_us" and "untraced_us" and the traced
    launches' average shader clock under "clock_mhz", C)."""
    import statistics
    import torch
    from paper_2506_11209_amd import inputs
    from paper_2506_11209_amd import wsgemm as w
    from paper_2506_11209_amd.workloads import unpack
    tm, tn, tk, stages, np_, nc, split = unpack(point)
    if Ad is None:
        A, B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
        Ad, Bd = A.cuda(), B.cuda()
    g = w.WsGemm(wl.M, wl.N, wl.K, (tm, tn, tk), stages, np_, nc, wl.dtype, load_path, split=split)
    try:
        wgs = min(wgs, g.info.grid)
        iters = g.info.rounds * g.info.iters
        buf = torch.zeros((wgs, iters, len(EVENTS)), dtype=torch.int32, device="cuda")
        C = torch.empty((wl.M, wl.N), dtype=torch.float32, device="cuda")
        for _ in range(warmup):
            g(Ad, Bd, C)

        def timed():
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g(Ad, Bd, C)
            e1.record()
            e1.synchronize()
            return e0.elapsed_time(e1) * 1e3

        untraced, traced, clocks = [], [], []
        for _ in range(max(1, pairs)):
            w.ws_gemm_set_trace(g._h, None)
            untraced.append(timed())  # the same launch untraced, for the tracing overhead
            s = w.ws_gemm_set_trace(g._h, buf.data_ptr(), buf.numel() * 4, wgs, iters)
            if s != w.WS_OK:
                raise w.WsGemmError("ws_gemm_set_trace", s)
            g.clock_mhz()
            traced.append(timed())
            clocks.append(g.clock_mhz()[0])
        if g.sync_status() != w.WS_OK:
            raise RuntimeError("traced run timed out")
        rec = buf.cpu().numpy().view(np.uint32)
        plan = g.info.as_dict()
        plan["traced_us"] = statistics.median(traced)
        plan["untraced_us"] = statistics.median(untraced)
        plan["clock_mhz"] = statistics.median(c for c in clocks if c) if any(clocks) else None
    finally:
        g.close()
    return rec, plan, C


def rel(rec_wg, n_iters):
    """Stamps of one workgroup relative to its first event, as int64 (wrap-safe)."""
    r = rec_wg[:n_iters].astype(np.int64)
    base = r[0, 0]
    out = (r - base) % (1 << 32)
    out[out > (1 << 31)] -= (1 << 32)
    return out


def summarize(rec, plan):
    """Per traced workgroup: medians of the per-K-iteration quantities in
    shader clocks, and the same in us at the clock measured over the traced
    launch (when its duration is known)."""
    S = plan["iters"]
    res = []
    for g in range(rec.shape[0]):
        tiles = len(range(g, plan["tiles"], plan["grid"]))
        n = tiles * S
        t = rel(rec[g], n)
        ia, ib, la, lb, ready, mma, relz = (t[:, i] for i in range(7))
        period = np.diff(mma)
        wait = ready[1:] - relz[:-1]  # consumer stall between releasing q-1 and seeing q
        ep = [t[k * S + S - 1, 7] - relz[k * S + S - 1] for k in range(tiles)]
        res.append({
            "wg": g, "iters": int(n),
            "period_median": float(np.median(period)),
            "load_a_median": float(np.median(la - ia)), "load_b_median": float(np.median(lb - ib)),
            "wait_mean": float(np.mean(np.maximum(wait, 0))),
            "wait_frac_iters": float(np.mean(wait > 200)),
            "ready_to_mma_median": float(np.median(mma - ready)),
            "epilogue_median": float(np.median(ep)) if ep else 0.0,
            "total_cycles": float(mma[-1] - mma[0]),
        })
    if res and (plan.get("clock_mhz") or plan.get("traced_us")):
        # the launch's measured clock, else: the traced workgroups run from
        # the first to the last round
        clock = plan.get("clock_mhz") or float(np.median([r["total_cycles"] for r in res])) / plan["traced_us"]
        for r in res:
            r["clock_ghz"] = clock / 1e3
            for k in ("period_median", "load_a_median", "load_b_median", "wait_mean", "ready_to_mma_median",
                      "epilogue_median"):
                r[k.replace("_median", "").replace("_mean", "") + "_us"] = r[k] / clock
    return res


def model_comparison(wl, point, rec, plan, clock_mhz, load_path="registers", steps=20, warmup=10):
    """The paper's event recurrences (Section 2.2, Eq. 1-3, persistent
    schedule) with this launch's own per-K-iteration costs, measured by the
    calibration kernels (Section 4.2: load-only A, load-only B and math-only
    kernels of the same launch, from two values of K), set against the
    traced workgroups' measured events.  Times in us; the traces' shader
    clocks are converted with the launch's measured clock."""
    import torch
    from paper_2506_11209_amd import calibrate as cal
    from paper_2506_11209_amd import wsgemm as w
    from paper_2506_11209_amd.workloads import split_of, unpack
    tm, tn, tk, P, np_, nc, split = unpack(point)
    tile = (tm, tn, tk)
    mn = min(wl.M, wl.N)
    A = torch.empty((mn, cal.K_PAIR[1]), dtype=torch.bfloat16, device="cuda").normal_()
    B = torch.empty((cal.K_PAIR[1], mn), dtype=torch.bfloat16, device="cuda").normal_()
    C = torch.empty((mn, mn), dtype=torch.float32, device="cuda")
    costs = {}
    for kind in ("load_a", "load_b", "math"):
        costs[kind], _ = cal.per_iteration_us(kind, tile, np_, load_path, (A, B, C), steps, warmup, nc, split, P)
    t_init, t_epi_kernel, rounds = cal.fixed_costs_us(mn, tile, np_, load_path, A, B, C, warmup, nc, split, P)
    t_epi = max(0.0, (t_epi_kernel - t_init) / rounds)
    S, W = plan["iters"], plan["rounds"]
    opts = w.model_options(two_dma=(split_of(point) == 2), persistent=True)
    st, s_a, s_b, s_m = w.ws_model_events(S, W, P, costs["math"], costs["load_a"], costs["load_b"], t_epi, opts)
    if st != w.WS_OK:
        raise RuntimeError("ws_model_events: %s" % w.ws_gemm_status_str(st))
    s_a, s_b, s_m = (np.asarray(x) for x in (s_a, s_b, s_m))
    per_us = clock_mhz  # shader clocks per us
    rows = []
    for g in range(rec.shape[0]):
        tiles = len(range(g, plan["tiles"], plan["grid"]))
        n = tiles * S
        t = rel(rec[g], n).astype(np.float64) / per_us
        ia, ib, mma = t[:, 0], t[:, 1], t[:, 5]
        m_sm = s_m[:n] - s_m[0]
        rows.append({
            "wg": g, "iters": int(n),
            "measured_dSm_median_us": float(np.median(np.diff(mma))),
            "model_dSm_median_us": float(np.median(np.diff(m_sm))),
            "measured_Sm_last_us": float(mma[n - 1] - mma[0]),
            "model_Sm_last_us": float(m_sm[n - 1]),
            "measured_Sm_minus_Sa_median_us": float(np.median(mma - ia)),
            "model_Sm_minus_Sa_median_us": float(np.median(s_m[:n] - s_a[:n])),
            "measured_Sm_minus_Sb_median_us": float(np.median(mma - ib)),
            "model_Sm_minus_Sb_median_us": float(np.median(s_m[:n] - s_b[:n])),
        })
    return {"t_math_us": costs["math"], "t_load_a_us": costs["load_a"], "t_load_b_us": costs["load_b"],
            "t_init_us": t_init, "t_epilogue_us": t_epi, "clock_mhz": clock_mhz, "workgroups": rows}


def main(argv=None):
    from paper_2506_11209_amd.workloads import WORKLOADS
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="gemm_8192x8192x8192_bf16_normal", choices=sorted(WORKLOADS))
    ap.add_argument("--point", default="256x128x64x3x4x4")
    ap.add_argument("--wgs", type=int, default=4)
    ap.add_argument("--load-path", default="registers", choices=("registers", "dma"))
    ap.add_argument("--dump", default=None, help="write the raw records (.npy)")
    ap.add_argument("--warmup", type=int, default=20, help="untraced launches before the traced one")
    ap.add_argument("--pairs", type=int, default=10, help="untraced / traced launch pairs (medians)")
    ap.add_argument("--model", action="store_true",
                    help="also set the measured events against the paper's recurrences with this launch's "
                         "calibrated costs")
    a = ap.parse_args(argv)
    wl = WORKLOADS[a.workload]
    from paper_2506_11209_amd.workloads import parse_point
    point = parse_point(a.point)
    rec, plan, _ = run_traced(wl, point, a.wgs, load_path=a.load_path, warmup=a.warmup, pairs=a.pairs)
    if a.dump:
        np.save(a.dump, rec)
    print(json.dumps({"point": a.point, "traced_us": plan.get("traced_us"),
                      "untraced_us": plan.get("untraced_us"), "traced_clock_mhz": plan.get("clock_mhz"),
                      "overhead": (plan["traced_us"] / plan["untraced_us"] - 1.0)
                      if plan.get("untraced_us") else None}))
    for r in summarize(rec, plan):
        print(json.dumps(r))
    if a.model:
        print(json.dumps(model_comparison(wl, point, rec, plan, plan["clock_mhz"], a.load_path)))


if __name__ == "__main__":
    main()
