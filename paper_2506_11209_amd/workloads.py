"""The GEMM workloads exercised by the tests, the sweep and the benchmark.

Each entry names a problem shape, the operand distribution and seed, and the
launch points (tile tuple, stage depth, producer/consumer waves) run on it.
A launch point is ``(tile_m, tile_n, tile_k, stages, producer_waves,
consumer_waves)`` or, where the wave counts do not imply it, the same with a
seventh entry: the split (DMA warps per MATH warp, 1 or 2).
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


def unpack(point):
    """(tm, tn, tk, stages, producer_waves, consumer_waves, split) of a launch
    point; split 0 (implied by the wave counts) when the point has none."""
    tm, tn, tk, stages, np_, nc = point[:6]
    return tm, tn, tk, stages, np_, nc, (point[6] if len(point) > 6 else 0)


def split_of(point) -> int:
    """DMA warps per MATH warp of a launch point (0: the synchronous kernel)."""
    _, _, _, _, np_, nc, split = unpack(point)
    if np_ == 0:
        return 0
    return split or (2 if np_ == 2 * nc else 1)


def point_key(point) -> str:
    """Text form of a launch point: TMxTNxTKxSTAGESxNPxNC[xSPLIT]."""
    return "x".join(map(str, point))


def parse_point(text: str):
    p = tuple(int(x) for x in text.split("x"))
    if len(p) not in (6, 7):
        raise ValueError("a launch point is TMxTNxTKxSTAGESxNPxNC[xSPLIT]: %r" % text)
    return p


def _sweep_8192():
    pts = []
    for tile in ((64, 64, 64), (128, 128, 32), (128, 256, 32), (256, 128, 64)):
        for stages in (2, 3, 4):
            for split in (1, 2):
                pts.append(tile + (stages, 4 * split, 4))
            # 2:1 at the 1:1 wave count: two groups of two producer waves
            pts.append(tile + (stages, 4, 4, 2))
    # eight consumer waves (two per SIMD) and four producer waves on 256 x 256
    # tiles: 1:1 and 2:1 (two groups of two)
    for tk, depths in ((64, (2,)), (32, (2, 3, 4))):
        for stages in depths:
            for split in (1, 2):
                pts.append((256, 256, tk, stages, 4, 8, split))
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
        # small integers at the headline size: every element of C is exact
        Workload("gemm_8192x8192x8192_bf16_int4", 8192, 8192, 8192, "bf16", "int4", 33, True,
                 ((256, 256, 64, 2, 4, 8, 1), (256, 128, 64, 3, 4, 4))),
        Workload("gemm_16384x256x8192_bf16_uniform", 16384, 256, 8192, "bf16", "uniform", 4, False,
                 ((128, 64, 64, 4, 8, 4),)),
        Workload("gemm_2048x2048x32768_bf16_normal_k", 2048, 2048, 32768, "bf16", "normal_k", 5,
                 False, ((128, 128, 64, 4, 4, 4), (128, 128, 64, 4, 8, 4))),
    )
}
