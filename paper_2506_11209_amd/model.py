"""Host side of the performance model: calibrated parameters and predictions.

The model itself (Section 2, Eq. 1-3, and the execution simulator of Section
3.1) runs in the library (``ws_model_predict`` / ``ws_model_events``); this
module holds the calibration fit of Section 4.2 and marshals parameters.
"""
from __future__ import annotations

import json
from dataclasses import asdict, dataclass

from paper_2506_11209_amd import wsgemm as w


@dataclass
class Params:
    """Machine parameters of the model, per workgroup (times in us)."""
    t_init: float
    t_epilogue: float
    compute_throughput: float  # multiply-accumulates per us
    compute_latency: float
    load_throughput: float     # elements per us
    load_latency: float

    def c(self) -> w.ws_model_params:
        return w.ws_model_params(self.t_init, self.t_epilogue, self.compute_throughput,
                                 self.compute_latency, self.load_throughput, self.load_latency)


def two_point_fit(work1: float, t1: float, work2: float, t2: float):
    """Section 4.2: throughput from the difference of two measurements of
    different work, startup latency as the remainder of the first one."""
    if t1 == t2:
        raise ValueError("the two calibration points must differ in time")
    thr = (work1 - work2) / (t1 - t2)
    return thr, t1 - work1 / thr


def predict(M, N, K, tile, stages, slots, params: Params, two_dma=False, persistent=True,
            finish_math=False) -> dict:
    tm, tn, tk = tile
    s, r = w.ws_model_predict(M, N, K, tm, tn, tk, stages, slots, params.c(),
                              w.model_options(two_dma, persistent, finish_math))
    if s != w.WS_OK:
        raise ValueError("ws_model_predict: %s" % w.ws_gemm_status_str(s))
    return r.as_dict()


def predict_costs(M, N, K, tile, stages, slots, params: Params, t_math, t_load_a, t_load_b,
                  two_dma=False, persistent=True, finish_math=False) -> dict:
    """Prediction from measured per-K-iteration costs of this configuration."""
    tm, tn, tk = tile
    s, r = w.ws_model_predict_costs(M, N, K, tm, tn, tk, stages, slots, t_math, t_load_a, t_load_b,
                                    params.c(), w.model_options(two_dma, persistent, finish_math))
    if s != w.WS_OK:
        raise ValueError("ws_model_predict_costs: %s" % w.ws_gemm_status_str(s))
    return r.as_dict()


def load_calibration(path: str) -> dict:
    """{(split, load_path): Params} from a file written by calibrate.py."""
    with open(path) as f:
        doc = json.load(f)
    out = {}
    for rec in doc["calibrations"]:
        out[(rec["split"], rec["load_path"])] = Params(**rec["params"])
    return out


def table_key(split: int, load_path: str, tile, consumer_waves: int = 4):
    """Key of a tile's measured costs in load_cost_table's result: four-consumer
    launches by (split, load path, tile), others with the consumer count too."""
    tile = tuple(tile)
    return (split, load_path, tile) if consumer_waves == 4 else (split, load_path, tile, consumer_waves)


def load_cost_table(path: str) -> dict:
    """{table_key(...): (t_math, t_load_a, t_load_b)} from a calibration file
    written with --table.

    Two DMA groups load A and B concurrently, so each takes the time measured
    with only its own tile loaded.  One DMA group issues both tiles of a
    K-iteration back to back; its measured time for both is split between
    T_LOAD-A and T_LOAD-B in proportion to the elements, so that the
    sequential loads of Eq. 1-2 add up to the measured time."""
    with open(path) as f:
        doc = json.load(f)
    out = {}
    for rec in doc["calibrations"]:
        for row in rec.get("table", []):
            tm, tn, tk = row["tile"]
            if rec["split"] == 2:
                la, lb = row["t_load_a"], row["t_load_b"]
            else:
                la = row["t_load_ab"] * tm / (tm + tn)
                lb = row["t_load_ab"] * tn / (tm + tn)
            out[table_key(rec["split"], rec["load_path"], (tm, tn, tk), row.get("consumer_waves", 4))] = (
                row["t_math"], la, lb)
    return out


def params_dict(p: Params) -> dict:
    return asdict(p)


# -- configuration optimizer (Section 3.2, by exhaustive search) ---------------

def compiled_configs(dtype="bf16", splits=(1, 2), consumer_waves=(4, 8)):
    """(tile, producer_waves, consumer_waves, split) of every compiled
    specialised GEMM kernel of the given dtype (the library is built from
    build.instances()) in the arrangements the calibration covers: split
    groups of four producer waves with four consumer waves, and four producer
    waves in one or two groups with eight consumer waves."""
    from paper_2506_11209_amd.build import MODE_GEMM, instances
    want_bf16 = 1 if dtype == "bf16" else 0
    out = set()
    for (tm, tn, tk, nc, np_, split, bf16, trace, mode, general) in instances():
        if bf16 != want_bf16 or trace or general or mode != MODE_GEMM or split not in splits:
            continue
        if nc in consumer_waves and ((nc == 4 and np_ == 4 * split) or (nc == 8 and np_ == 4)):
            out.add(((tm, tn, tk), np_, nc, split))
    return sorted(out)


def candidates(M, N, K, dtype="bf16", splits=(1, 2), stages=range(2, 9), num_cus=256,
               load_path="registers", consumer_waves=(4, 8)):
    """Launchable (tile, stages, producer_waves, consumer_waves, slots, split)
    for this problem: compiled, ring fits in LDS, tiles divide the problem.
    `slots` is the planned grid (workgroups that run at once)."""
    out = []
    for tile, np_, nc, split in compiled_configs(dtype, splits, consumer_waves):
        for P in stages:
            cfg = w.config(tile, P, np_, nc, dtype, load_path, split)
            s, info = w.ws_gemm_plan(M, N, K, cfg, num_cus, 0)
            if s == w.WS_OK:
                out.append((tile, P, np_, nc, info.grid, split))
    return out


def optimize(M, N, K, params_by_split: dict, cands, objective="time", persistent=True,
             table: dict | None = None, load_path="registers"):
    """Rank candidate launches by predicted time (objective "time", Section 3.2's
    first goal) or by predicted total MATH wait (second goal; ties broken by
    time, then by the deeper ring).  params_by_split: {1: Params, 2: Params}.  With `table` (from
    load_cost_table), tiles that were measured use their own costs; the others
    the fitted linear costs.  The fits are calibrated on four-consumer kernels:
    a candidate with another consumer count is ranked only with its own
    measured costs, and left out without them.  A candidate is (tile, stages,
    producer_waves, consumer_waves, slots[, split]); split defaults to
    producer_waves / consumer_waves.  Returns a list of dicts, best first."""
    rows = []
    for c in cands:
        tile, P, np_, nc, slots = c[:5]
        split = c[5] if len(c) > 5 else np_ // nc
        costs = table.get(table_key(split, load_path, tile, nc)) if table else None
        if costs is None and nc != 4:
            continue
        if costs is not None:
            r = predict_costs(M, N, K, tile, P, slots, params_by_split[split], *costs,
                              two_dma=(split == 2), persistent=persistent)
        else:
            r = predict(M, N, K, tile, P, slots, params_by_split[split], two_dma=(split == 2),
                        persistent=persistent)
        rows.append({"tile": tile, "stages": P, "producer_waves": np_, "consumer_waves": nc, "split": split,
                     "slots": slots, "time_us": r["total_us"], "wait_us": r["wait_us"],
                     "costs": "table" if costs is not None else "fit"})
    # Ties (the model gives every ring depth the same time once the pipeline
    # is compute- or DMA-bound) go to the deeper ring: it is never slower in
    # the model and hides latency the model does not represent.
    if objective == "time":
        rows.sort(key=lambda r: (r["time_us"], r["wait_us"], -r["stages"]))
    else:
        rows.sort(key=lambda r: (r["wait_us"], r["time_us"], -r["stages"]))
    return rows
