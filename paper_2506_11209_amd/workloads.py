"""The GEMM workloads exercised by the tests, the sweep and the benchmark.

Each entry names a problem shape, the operand distribution and seed, and the
launch points (tile tuple, stage depth, producer/consumer waves) run on it.
A launch point is ``(tile_m, tile_n, tile_k, stages, producer_waves,
consumer_waves)``.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    dtype: str
    dist: str
    seed: int
    exact: bool  # small-integer operands: results must be bit-exact
    points: tuple = field(default_factory=tuple)

    @property
    def flops(self) -> float:
        return 2.0 * self.M * self.N * self.K

    @property
    def bytes(self) -> float:
        esz = 2
        return esz * (self.M * self.K + self.K * self.N) + 4.0 * self.M * self.N


def _sweep_8192():
    pts = []
    for tile in ((64, 64, 64), (128, 128, 32), (128, 256, 32), (256, 128, 64)):
        for stages in (2, 3, 4):
            for split in (1, 2):
                pts.append(tile + (stages, 4 * split, 4))
    # the synchronous baseline (no producer waves): ring depth 1 and 2
    for tile in ((128, 128, 32), (128, 256, 32), (256, 128, 64), (256, 256, 64)):
        for stages in (1, 2):
            pts.append(tile + (stages, 0, 4))
    return tuple(pts)


WORKLOADS = {
    w.name: w
    for w in (
        Workload("gemm_256x256x256_f16_int4", 256, 256, 256, "f16", "int4", 1, True,
                 ((64, 64, 32, 2, 1, 1),)),
        Workload("gemm_4096x4096x4096_bf16_normal", 4096, 4096, 4096, "bf16", "normal", 2, False,
                 ((128, 128, 32, 3, 4, 4),)),
        Workload("gemm_8192x8192x8192_bf16_normal", 8192, 8192, 8192, "bf16", "normal", 3, False,
                 _sweep_8192()),
        Workload("gemm_16384x256x8192_bf16_uniform", 16384, 256, 8192, "bf16", "uniform", 4, False,
                 ((128, 64, 64, 4, 8, 4),)),
        Workload("gemm_2048x2048x32768_bf16_normal_k", 2048, 2048, 32768, "bf16", "normal_k", 5,
                 False, ((128, 128, 64, 4, 4, 4), (128, 128, 64, 4, 8, 4))),
    )
}
