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


def load_cost_table(path: str) -> dict:
    """{(split, load_path, (tm, tn, tk)): (t_math, t_load_a, t_load_b)} from
    a calibration file written with --table.

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
            out[(rec["split"], rec["load_path"], (tm, tn, tk))] = (row["t_math"], la, lb)
    return out


def params_dict(p: Params) -> dict:
    return asdict(p)
