"""Summaries of rocprofv3 result databases (rocpd SQLite) as short text.

    python -m paper_2506_11209_amd.profsummary trace  DB [--kernel SUBSTR] [--skip N]
    python -m paper_2506_11209_amd.profsummary counters DB [--kernel SUBSTR] [--group G --points JSONL]
    python -m paper_2506_11209_amd.profsummary sweeptable SWEEP_JSONL COUNTERS_JSONL... [--scales F,W]
    python -m paper_2506_11209_amd.profsummary traffic FETCH_DB WRITE_DB CAL_FETCH_DB CAL_WRITE_DB \
        --kernel SUBSTR --point KEY [--workload NAME] [--dtype bf16] [--copy-mib 1024]

`trace`: per-kernel call count, mean / median / min duration (us), from
`rocprofv3 --kernel-trace` (with `--group G`: the matching dispatches in
launch order cut into consecutive runs of G, one line per run, for programs
that time one case after another).  `counters`: per-kernel mean of each collected
counter over its dispatches (instances summed per dispatch), from
`rocprofv3 --pmc ...`.  `traffic`: HBM bytes per launch of a kernel from
FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by bytes-moved /
counter-reading of the known-size copy run by
`python -m paper_2506_11209_amd.hbm_calibrate`; printed as the JSON record
bench.py reads (tagged with the fingerprint of the kernel's machine code).
"""
from __future__ import annotations

import argparse
import collections
import sqlite3
import statistics


def kernel_durations(db_path: str, kernel: str | None = None, skip: int = 0):
    """Durations (us) per kernel name in dispatch order, the first `skip`
    dispatches of each kernel (the untimed warm-up launches) left out."""
    db = sqlite3.connect(db_path)
    rows = db.execute("select name, duration from kernels order by start").fetchall()
    out = collections.defaultdict(list)
    for name, dur in rows:
        if kernel is None or kernel in name:
            out[name].append(dur / 1e3)  # ns -> us
    return {k: v[skip:] for k, v in out.items() if len(v) > skip}


def dispatch_runs(db_path: str, kernel: str | None, group: int, skip: int = 0):
    """Matching dispatches in launch order, cut into consecutive runs of
    `group`; each run as (kernel name, durations in us after its first
    `skip`)."""
    db = sqlite3.connect(db_path)
    rows = [(n, d / 1e3) for n, d in db.execute("select name, duration from kernels order by start")
            if kernel is None or kernel in n]
    return [(rows[i][0], [d for _, d in rows[i:i + group]][skip:]) for i in range(0, len(rows), group)]


def counter_means(db_path: str, kernel: str | None = None):
    db = sqlite3.connect(db_path)
    rows = db.execute("select name, dispatch_id, counter_name, counter_value from pmc_events").fetchall()
    per = collections.defaultdict(float)
    for name, did, cn, cv in rows:
        if kernel is None or kernel in name:
            per[(name, did, cn)] += cv
    agg = collections.defaultdict(list)
    for (name, did, cn), v in per.items():
        agg[(name, cn)].append(v)
    return {k: (statistics.fmean(v), len(v)) for k, v in agg.items()}


def counter_runs(db_path: str, kernel: str | None, group: int, skip: int = 0):
    """Matching dispatches in launch order, cut into consecutive runs of
    `group` (one per case of a program that runs its cases one after another,
    each `group` times); per run: (kernel name, {counter: mean over the run's
    dispatches after its first `skip`}, instances summed per dispatch)."""
    db = sqlite3.connect(db_path)
    rows = db.execute("select name, dispatch_id, counter_name, counter_value from pmc_events").fetchall()
    per = collections.defaultdict(float)
    names = {}
    for name, did, cn, cv in rows:
        if kernel is None or kernel in name:
            per[(did, cn)] += cv
            names[did] = name
    dids = sorted(names)
    out = []
    for i in range(0, len(dids), group):
        run = dids[i:i + group][skip:]
        counters = sorted({cn for (d, cn) in per if d in run})
        out.append((names[dids[i]], {cn: statistics.fmean(per[(d, cn)] for d in run) for cn in counters}))
    return out


def _mean_counter(db_path, name_part, counter):
    vals = [v for (n, cn), (v, _) in counter_means(db_path).items() if name_part in n and cn == counter]
    if not vals:
        raise SystemExit("no %s for %s in %s" % (counter, name_part, db_path))
    return vals[0]


def traffic(fetch_db, write_db, cal_fetch_db, cal_write_db, kernel, point, copy_mib, workload, dtype):
    import json
    import os
    import sys
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from bench import WORKLOAD, kernel_fingerprint
    from paper_2506_11209_amd.workloads import parse_point
    point_t = parse_point(point.split("/")[0])
    copy_bytes = copy_mib * (1 << 20)
    f_scale = copy_bytes / (_mean_counter(cal_fetch_db, "copyBuffer", "FETCH_SIZE") * 1024)
    w_scale = copy_bytes / (_mean_counter(cal_write_db, "copyBuffer", "WRITE_SIZE") * 1024)
    fetch = _mean_counter(fetch_db, kernel, "FETCH_SIZE")
    write = _mean_counter(write_db, kernel, "WRITE_SIZE")
    rec = {"kernel": kernel, "workload": workload or WORKLOAD, "point": point,
           "kernel_fingerprint": kernel_fingerprint(point_t, dtype),
           "fetch_size_kib": fetch, "write_size_kib": write,
           "fetch_scale_bytes_per_kib": f_scale * 1024, "write_scale_bytes_per_kib": w_scale * 1024,
           "traffic_bytes_per_launch": fetch * 1024 * f_scale + write * 1024 * w_scale}
    print(json.dumps(rec, indent=1))


def sweep_table(timing_jsonl: str, counter_jsonls: list, fetch_scale: float, write_scale: float,
                cus: int = 256, xcds: int = 8, load_path: str = "registers") -> str:
    """Markdown table: one row per launch point of a sweep, joining the
    timing run (sweep.py JSON lines) with the per-point counter runs
    (`counters --group --points` output) of the same points.
      MFMA busy  SQ_VALU_MFMA_BUSY_CYCLES per SIMD / GRBM_GUI_ACTIVE per XCD
      LDS busy   SQ_LDS_IDX_ACTIVE per CU / GRBM_GUI_ACTIVE per XCD
      LDS wait   SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES (wave cycles waiting to
                 issue an LDS instruction)
      L2 hit     TCC_HIT / (TCC_HIT + TCC_MISS)
      fetch, write  FETCH_SIZE, WRITE_SIZE scaled by a known-size copy's
                 bytes per counted KiB: L2-to-fabric request bytes (memory
                 side, including Infinity Cache hits), in GB per launch."""
    import json
    timing = {}
    with open(timing_jsonl) as f:
        for r in map(json.loads, f):
            timing[r["point"]] = r
    counters = collections.defaultdict(dict)
    for path in counter_jsonls:
        with open(path) as f:
            for r in map(json.loads, f):
                counters[r["point"]].update(r["counters"])
    simds = 4 * cus
    lines = ["| point | TFLOP/s | clock MHz | MFMA busy | LDS busy | LDS wait | bank conflicts | L2 hit | "
             "fetch GB | write GB |", "|---|---|---|---|---|---|---|---|---|---|"]
    for key, r in timing.items():
        if not key.endswith("/" + load_path):
            continue
        c = counters.get(key, {})
        if r.get("status") != "ok":
            lines.append("| %s | %s | | | | | | | | |" % (key, r.get("status")))
            continue
        grbm = c.get("GRBM_GUI_ACTIVE")
        per_xcd = grbm / xcds if grbm else None

        def frac(num, den):
            return "%.1f %%" % (100.0 * num / den) if num is not None and den else "-"
        mfma = c.get("SQ_VALU_MFMA_BUSY_CYCLES")
        lds = c.get("SQ_LDS_IDX_ACTIVE")
        hit, miss = c.get("TCC_HIT"), c.get("TCC_MISS")
        lines.append("| %s | %.0f | %s | %s | %s | %s | %s | %s | %s | %s |" % (
            key, r["tflops"], "%.0f" % r["clock_mhz"] if r.get("clock_mhz") else "-",
            frac(mfma / simds if mfma is not None else None, per_xcd),
            frac(lds / cus if lds is not None else None, per_xcd),
            frac(c.get("SQ_WAIT_INST_LDS"), c.get("SQ_WAVE_CYCLES")),
            "%.0f" % c["SQ_LDS_BANK_CONFLICT"] if "SQ_LDS_BANK_CONFLICT" in c else "-",
            frac(hit, (hit + miss) if hit is not None and miss is not None else None),
            "%.2f" % (c["FETCH_SIZE"] * fetch_scale / 1e9) if "FETCH_SIZE" in c else "-",
            "%.2f" % (c["WRITE_SIZE"] * write_scale / 1e9) if "WRITE_SIZE" in c else "-"))
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("mode", choices=("trace", "counters", "traffic", "sweeptable"))
    ap.add_argument("db", nargs="+")
    ap.add_argument("--kernel", default=None)
    ap.add_argument("--point", default=None)
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--workload", default=None, help="traffic: workload the counters ran (default: the bench's)")
    ap.add_argument("--dtype", default="bf16", help="traffic: operand dtype of the kernel")
    ap.add_argument("--skip", type=int, default=0, help="trace: leading dispatches per kernel (or run) to drop")
    ap.add_argument("--last", type=int, default=0,
                    help="trace: keep only the last N dispatches per kernel (a program's timed launches after "
                         "a warm-up of varying length)")
    ap.add_argument("--group", type=int, default=0, help="trace / counters: dispatches per consecutive run")
    ap.add_argument("--points", default=None,
                    help="counters --group: the sweep's JSON lines, to label each run with its launch point")
    ap.add_argument("--scales", default="2047.9,1024.0",
                    help="sweeptable: FETCH_SIZE and WRITE_SIZE bytes per counted KiB (from a copy run)")
    a = ap.parse_args(argv)
    if a.mode == "sweeptable":
        fs, ws = (float(x) for x in a.scales.split(","))
        print(sweep_table(a.db[0], a.db[1:], fs, ws))
        return
    if a.mode == "traffic":
        traffic(*a.db[:4], a.kernel, a.point, a.copy_mib, a.workload, a.dtype)
        return
    a.db = a.db[0]
    if a.mode == "trace" and a.group > 0:
        for i, (name, d) in enumerate(dispatch_runs(a.db, a.kernel, a.group, a.skip)):
            if d:
                print("run %-3d %-64s n=%-4d mean_us=%.2f median_us=%.2f min_us=%.2f" % (
                    i, name[:64], len(d), statistics.fmean(d), statistics.median(d), min(d)))
    elif a.mode == "trace":
        durs = kernel_durations(a.db, a.kernel, a.skip)
        if a.last > 0:
            durs = {k: v[-a.last:] for k, v in durs.items()}
        for name, d in sorted(durs.items(), key=lambda x: -sum(x[1])):
            print("%-72s calls=%-5d mean_us=%.2f median_us=%.2f min_us=%.2f" % (
                name[:72], len(d), statistics.fmean(d), statistics.median(d), min(d)))
    elif a.group > 0:
        import json
        labels = []
        if a.points:
            with open(a.points) as f:
                labels = [r["point"] for r in map(json.loads, f) if r.get("status") == "ok"]
        for i, (name, c) in enumerate(counter_runs(a.db, a.kernel, a.group, a.skip)):
            label = labels[i] if i < len(labels) else "run %d" % i
            print(json.dumps({"point": label, "kernel": name, "counters": c}))
    else:
        for (name, cn), (mean, n) in sorted(counter_means(a.db, a.kernel).items()):
            print("%-72s %-32s mean=%.6g dispatches=%d" % (name[:72], cn, mean, n))


if __name__ == "__main__":
    main()
