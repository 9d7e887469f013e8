"""Device-side timing of library launches with HIP events.

Events are recorded on the same stream the kernel is launched on (torch's
current stream, whose handle is passed to ws_gemm_run), one pair per launch.
"""
from __future__ import annotations

import statistics
import time

import torch


def time_launches(launch, steps: int, warmup: int):
    """Run ``launch()`` warmup + steps times; return per-launch device ms and
    the wall-clock ms per step of the timed region (synchronised both sides)."""
    for _ in range(warmup):
        launch()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        starts[i].record()
        launch()
        ends[i].record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    dev = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    return dev, wall_ms


def summary(dev_ms):
    return {
        "mean_ms": statistics.fmean(dev_ms),
        "median_ms": statistics.median(dev_ms),
        "std_ms": statistics.pstdev(dev_ms) if len(dev_ms) > 1 else 0.0,
        "min_ms": min(dev_ms),
        "n": len(dev_ms),
    }
