"""Timing of the general kernel variant against the plain kernel.

    python -m paper_2506_11209_amd.variants_bench [--steps 30] [--warmup 10] [--out FILE]
                                                  [--point TMxTNxTKxSTAGESxNPxNC[xSPLIT]]

Cases (bf16 operands, by default tile 256x128x64, 3 stages, 4 producer + 4
consumer waves; --point another launch; register-staged producers, normal
inputs):
  * M = N = K = 8192 with the default epilogue (the plain kernel) and with
    epilogues that need the general variant: bf16 output, fp16 output, and
    alpha / beta with fp32 output (beta != 0 reads C);
  * shapes the tiles do not divide, next to the whole-tile shapes around
    them (general variant vs plain kernel).
One JSON line per case: device time per launch from HIP events on the
launch stream, TFLOP/s on the case's own 2 M N K.
"""
from __future__ import annotations

import argparse
import json
import sys

import torch

from paper_2506_11209_amd import inputs
from paper_2506_11209_amd import wsgemm as w
from paper_2506_11209_amd.timing import summary, time_launches

DEFAULT_POINT = (256, 128, 64, 3, 4, 4)
TORCH_OUT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}

# (name, (M, N, K), (alpha, beta, out dtype))
CASES = [
    ("8192 plain", (8192, 8192, 8192), (1.0, 0.0, "f32")),
    ("8192 out bf16", (8192, 8192, 8192), (1.0, 0.0, "bf16")),
    ("8192 out f16", (8192, 8192, 8192), (1.0, 0.0, "f16")),
    ("8192 alpha 2 beta 0 f32", (8192, 8192, 8192), (2.0, 0.0, "f32")),
    ("8192 alpha 1 beta 1 f32", (8192, 8192, 8192), (1.0, 1.0, "f32")),
    ("7936 whole", (7936, 7936, 7936), (1.0, 0.0, "f32")),
    ("8000 ragged", (8000, 8000, 8000), (1.0, 0.0, "f32")),
    ("4096 whole", (4096, 4096, 4096), (1.0, 0.0, "f32")),
    ("4100x4104x4104 ragged", (4100, 4104, 4104), (1.0, 0.0, "f32")),
]


_operands = {}


def operands(M, N, K):
    """Device operands of one shape, drawn once per shape."""
    if (M, N, K) not in _operands:
        _operands.clear()
        A, B = inputs.make_operands(M, N, K, "bf16", "normal", 1)
        _operands[(M, N, K)] = (A.cuda(), B.cuda())
    return _operands[(M, N, K)]


def measure(name, shape, epi, steps, warmup, point=DEFAULT_POINT):
    from paper_2506_11209_amd.workloads import unpack
    tm, tn, tk, stages, np_, nc, split = unpack(point)
    M, N, K = shape
    alpha, beta, out = epi
    Ad, Bd = operands(M, N, K)
    C = torch.zeros((M, N), dtype=TORCH_OUT[out], device="cuda")
    g = w.WsGemm(M, N, K, (tm, tn, tk), stages, np_, nc, "bf16", split=split)
    try:
        g.set_epilogue(alpha, beta, out)
        stream = torch.cuda.current_stream()
        a, b, c = Ad.data_ptr(), Bd.data_ptr(), C.data_ptr()
        dev, _ = time_launches(lambda: g.run_ptrs(a, b, c, stream.cuda_stream), steps, warmup)
        st = g.sync_status()
        if st != w.WS_OK:
            raise RuntimeError("%s: %s" % (name, w.ws_gemm_status_str(st)))
        s = summary(dev)
        return {"case": name, "point": "x".join(map(str, point)), "M": M, "N": N, "K": K, "alpha": alpha,
                "beta": beta, "out_dtype": out,
                "general": g.info.general, "ragged": g.info.ragged, "grid": g.info.grid,
                "mean_ms": round(s["mean_ms"], 5), "median_ms": round(s["median_ms"], 5),
                "tflops": round(2.0 * M * N * K / (s["median_ms"] * 1e-3) / 1e12, 1)}
    finally:
        g.close()


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--out", default=None)
    ap.add_argument("--point", default=None, help="TMxTNxTKxSTAGESxNPxNC[xSPLIT] (default 256x128x64x3x4x4)")
    a = ap.parse_args(argv)
    from paper_2506_11209_amd.workloads import parse_point
    point = parse_point(a.point) if a.point else DEFAULT_POINT
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    f = open(a.out, "a") if a.out else None
    for name, shape, epi in CASES:
        rec = measure(name, shape, epi, a.steps, a.warmup, point)
        line = json.dumps(rec)
        print(line, flush=True)
        if f:
            f.write(line + "\n")
            f.flush()
    return 0


if __name__ == "__main__":
    sys.exit(main())
