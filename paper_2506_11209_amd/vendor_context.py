"""The vendor library on the GEMM workloads, for context only.

    python -m paper_2506_11209_amd.vendor_context [--workload NAME ...] [--steps 30] [--warmup 20]

Times ``torch.mm`` (hipBLASLt) on the same seeded operands the benchmark
uses (``inputs.make_operands``), with a bf16 / fp16 result and with an fp32
result (``out_dtype=torch.float32``, the specialised kernel's output type),
by HIP events on the current stream after a time-based warm-up, and prints
one JSON line per workload and output type.  Nothing here is part of the
specialised kernel's path; the lines only place its figures beside what the
vendor library reaches on the same GPU.  Under ``rocprofv3 --kernel-trace``
or ``--pmc`` the same command gives the library kernels' durations and
counters.
"""
from __future__ import annotations

import argparse
import json
import sys

import torch

from paper_2506_11209_amd import inputs
from paper_2506_11209_amd.timing import summary, time_launches
from paper_2506_11209_amd.workloads import WORKLOADS


def measure(name: str, steps: int, warmup: int, min_warmup_s: float):
    wl = WORKLOADS[name]
    A, B = inputs.make_operands(wl.M, wl.N, wl.K, wl.dtype, wl.dist, wl.seed)
    A, B = A.cuda(), B.cuda()
    rows = []
    for out_name, kwargs, out_bytes in ((wl.dtype, {}, 2), ("f32", {"out_dtype": torch.float32}, 4)):
        def launch():
            torch.mm(A, B, **kwargs)
        dev, _ = time_launches(launch, steps, warmup, min_warmup_s=min_warmup_s)
        s = summary(dev)
        moved = 2.0 * (wl.M * wl.K + wl.K * wl.N) + out_bytes * wl.M * wl.N
        rows.append({"workload": name, "library": "torch.mm", "operands": wl.dtype, "output": out_name,
                     "mean_ms": s["mean_ms"], "median_ms": s["median_ms"], "n": s["n"],
                     "tflops": wl.flops / s["mean_ms"] / 1e9,
                     "gbs_algorithmic": moved / s["mean_ms"] / 1e6})
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", action="append", default=None,
                    help="workload name (repeatable; default: every workload)")
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--min-warmup-s", type=float, default=0.5)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        print("vendor_context needs a GPU", file=sys.stderr)
        return 2
    for name in args.workload or list(WORKLOADS):
        if name not in WORKLOADS:
            print("unknown workload %r" % name, file=sys.stderr)
            return 2
        for row in measure(name, args.steps, args.warmup, args.min_warmup_s):
            print(json.dumps(row), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
