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


def run_traced(wl, point, wgs=4, Ad=None, Bd=None, load_path="registers", warmup=0):
    """One traced launch after `warmup` untraced ones; returns (records [wgs,
    iters, 8] uint32, plan dict with the traced launch's duration in us under
    "traced_us", C)."""
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
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g(Ad, Bd, C)  # the same launch untraced, for the tracing overhead
        e1.record()
        torch.cuda.synchronize()
        untraced_us = e0.elapsed_time(e1) * 1e3
        s = w.ws_gemm_set_trace(g._h, buf.data_ptr(), buf.numel() * 4, wgs, iters)
        if s != w.WS_OK:
            raise w.WsGemmError("ws_gemm_set_trace", s)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g(Ad, Bd, C)
        e1.record()
        if g.sync_status() != w.WS_OK:
            raise RuntimeError("traced run timed out")
        rec = buf.cpu().numpy().view(np.uint32)
        plan = g.info.as_dict()
        plan["traced_us"] = e0.elapsed_time(e1) * 1e3
        plan["untraced_us"] = untraced_us
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
    if res and plan.get("traced_us"):
        # the traced workgroups run from the first to the last round
        clock = float(np.median([r["total_cycles"] for r in res])) / plan["traced_us"]  # clocks per us
        for r in res:
            r["clock_ghz"] = clock / 1e3
            for k in ("period_median", "load_a_median", "load_b_median", "wait_mean", "ready_to_mma_median",
                      "epilogue_median"):
                r[k.replace("_median", "").replace("_mean", "") + "_us"] = r[k] / clock
    return res


def main(argv=None):
    from paper_2506_11209_amd.workloads import WORKLOADS
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="gemm_8192x8192x8192_bf16_normal", choices=sorted(WORKLOADS))
    ap.add_argument("--point", default="256x128x64x3x4x4")
    ap.add_argument("--wgs", type=int, default=4)
    ap.add_argument("--load-path", default="registers", choices=("registers", "dma"))
    ap.add_argument("--dump", default=None, help="write the raw records (.npy)")
    ap.add_argument("--warmup", type=int, default=20, help="untraced launches before the traced one")
    a = ap.parse_args(argv)
    wl = WORKLOADS[a.workload]
    from paper_2506_11209_amd.workloads import parse_point
    point = parse_point(a.point)
    rec, plan, _ = run_traced(wl, point, a.wgs, load_path=a.load_path, warmup=a.warmup)
    if a.dump:
        np.save(a.dump, rec)
    print(json.dumps({"point": a.point, "traced_us": plan.get("traced_us"),
                      "untraced_us": plan.get("untraced_us")}))
    for r in summarize(rec, plan):
        print(json.dumps(r))


if __name__ == "__main__":
    main()
