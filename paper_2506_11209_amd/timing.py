"""Device-side timing of library launches with HIP events.

Events are recorded on the same stream the kernel is launched on (torch's
current stream, whose handle is passed to ws_gemm_run), one pair per launch.

Warm-up is by count and by time: the shader clock of an MI355X ramps over
the first tens of launches of a heavy kernel, so a fixed small count leaves
the timed region on a rising clock.  ``warm_up`` keeps launching until a
minimum time has passed and two consecutive batches agree.
"""
from __future__ import annotations

import statistics
import time

import torch


def warm_up(launch, min_launches: int, min_seconds: float = 0.5, batch: int = 10,
            tol: float = 0.01, max_seconds: float = 5.0) -> dict:
    """Launch at least ``min_launches`` times and for at least ``min_seconds``,
    then until the mean device time of the last batch of ``batch`` launches is
    within ``tol`` of the batch before it (at most ``max_seconds`` in all)."""
    for _ in range(min_launches):
        launch()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n = min_launches
    means = []
    while True:
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(batch):
            launch()
        e.record()
        e.synchronize()
        n += batch
        means.append(s.elapsed_time(e) / batch)
        elapsed = time.perf_counter() - t0
        settled = len(means) >= 2 and abs(means[-1] - means[-2]) <= tol * means[-2]
        if (elapsed >= min_seconds and settled) or elapsed >= max_seconds:
            return {"launches": n, "seconds": round(elapsed, 3), "settled": settled,
                    "last_batch_ms": [round(m, 5) for m in means[-2:]]}


def time_launches(launch, steps: int, warmup: int, min_warmup_s: float = 0.0,
                  with_warmup: bool = False, before_timed=None, between=None):
    """Warm up, then run ``launch()`` ``steps`` times; return the per-launch
    device ms and the wall-clock ms per step of the timed region
    (synchronised both sides), plus the warm-up record if ``with_warmup``.
    With ``min_warmup_s`` > 0 the warm-up is ``warm_up``'s (count, time and
    settled batches); otherwise it is ``warmup`` launches.  ``before_timed()``,
    if given, runs between the warm-up and the timed region (synchronised).
    ``between()``, if given, is enqueued before every timed launch, outside
    its pair of events (a cache flush for cold-cache timing); the wall-clock
    time per step then includes it."""
    if min_warmup_s > 0:
        wu = warm_up(launch, warmup, min_warmup_s)
    else:
        for _ in range(warmup):
            launch()
        wu = {"launches": warmup}
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    if before_timed is not None:
        before_timed()
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        if between is not None:
            between()
        starts[i].record()
        launch()
        ends[i].record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    dev = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    return (dev, wall_ms, wu) if with_warmup else (dev, wall_ms)


def summary(dev_ms):
    return {
        "mean_ms": statistics.fmean(dev_ms),
        "median_ms": statistics.median(dev_ms),
        "std_ms": statistics.pstdev(dev_ms) if len(dev_ms) > 1 else 0.0,
        "min_ms": min(dev_ms),
        "n": len(dev_ms),
    }
