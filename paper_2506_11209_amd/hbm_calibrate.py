"""Known-size copy used to calibrate HBM byte counters.

    python -m paper_2506_11209_amd.hbm_calibrate [--mib 1024] [--reps 3]

Copies a --mib MiB buffer into another (one torch copy kernel per
repetition): each launch reads and writes exactly that many bytes, more
than the last-level caches hold, so the FETCH_SIZE / WRITE_SIZE counters a
profiler reports for it give the scale factor between counter units and
bytes moved to and from HBM.
"""
import argparse

import torch


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--mib", type=int, default=1024)
    ap.add_argument("--reps", type=int, default=3)
    a = ap.parse_args()
    n = a.mib << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(a.reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print("copied %d bytes x %d launches" % (n, a.reps))


if __name__ == "__main__":
    main()
