"""Reference performance model of the warp-specialised GEMM -- TEST INFRASTRUCTURE ONLY.

A plain, slow transcription of the paper's performance model (Section 2,
"Performance Model") in its own order and notation, used to check the
library's model (``ws_model_*`` in the C ABI).  Indices are 1-based as in the
paper; lists carry an unused slot 0.

Readings taken where the paper is silent or self-contradictory:
  * the buffer capacity written "M" in Section 2.2 is the ring depth P;
  * for i <= P the release term S_m(i - P) + T_MATH does not exist (nothing
    has to be released yet), so it drops out of the max;
  * the round ends at S_m(S) + T_EPILOGUE as printed; `finish_math=True`
    adds the last T_MATH (the prose says the round ends when the last MATH
    finishes);
  * the two-DMA arrangement (two DMA warps per MATH warp, one per input
    tile) has no printed equations; here each DMA warp chains its own loads
    and waits for the same slot release, and MATH waits for both tiles;
  * `schedule="persistent"` models a persistent grid (the GPU kernel): one
    pipeline per workgroup runs through all W rounds back to back, and the
    epilogue of a tile delays the next tile's first MATH; the per-round
    schedule restarts the pipeline every round as Section 2.1 assumes.

Only the test suite may import this module.
"""
from __future__ import annotations

import math


def linear_costs(tm: int, tn: int, tk: int, compute_throughput: float, compute_latency: float,
                 load_throughput: float, load_latency: float):
    """Section 2.2 cost model: (T_MATH, T_LOAD-A, T_LOAD-B).

    Work is counted in elements as printed: T_M T_N T_K multiply-accumulates
    for MATH, T_M T_K elements of A and T_K T_N elements of B for the loads.
    """
    t_math = tm * tn * tk / compute_throughput + compute_latency
    t_load_a = tm * tk / load_throughput + load_latency
    t_load_b = tk * tn / load_throughput + load_latency
    return t_math, t_load_a, t_load_b


def events_one_dma(S: int, P: int, t_math: float, t_la: float, t_lb: float):
    """Eq. 1-3 (one DMA warp loads a_i, then b_i).  Returns (Sa, Sb, Sm)."""
    Sa = [0.0] * (S + 1)
    Sb = [0.0] * (S + 1)
    Sm = [0.0] * (S + 1)
    for i in range(1, S + 1):
        # Eq. 1: a_i starts after b_{i-1} has been loaded, and once the slot
        # of stage i - P has been released by MATH.
        if i == 1:
            Sa[i] = 0.0
        else:
            Sa[i] = Sb[i - 1] + t_lb
            if i - P >= 1:
                Sa[i] = max(Sa[i], Sm[i - P] + t_math)
        # Eq. 2: b_i starts after a_i has been loaded (and the same release).
        Sb[i] = Sa[i] + t_la
        if i - P >= 1:
            Sb[i] = max(Sb[i], Sm[i - P] + t_math)
        # Eq. 3: MATH of stage i starts after MATH of i - 1 and after b_i landed.
        Sm[i] = Sb[i] + t_lb
        if i >= 2:
            Sm[i] = max(Sm[i], Sm[i - 1] + t_math)
    return Sa, Sb, Sm


def events_two_dma(S: int, P: int, t_math: float, t_la: float, t_lb: float):
    """Two DMA warps per MATH warp, one loading A tiles and one loading B
    tiles, each chaining its own loads; MATH waits for both tiles."""
    Sa = [0.0] * (S + 1)
    Sb = [0.0] * (S + 1)
    Sm = [0.0] * (S + 1)
    for i in range(1, S + 1):
        Sa[i] = 0.0 if i == 1 else Sa[i - 1] + t_la
        Sb[i] = 0.0 if i == 1 else Sb[i - 1] + t_lb
        if i - P >= 1:
            Sa[i] = max(Sa[i], Sm[i - P] + t_math)
            Sb[i] = max(Sb[i], Sm[i - P] + t_math)
        Sm[i] = max(Sa[i] + t_la, Sb[i] + t_lb)
        if i >= 2:
            Sm[i] = max(Sm[i], Sm[i - 1] + t_math)
    return Sa, Sb, Sm


def events_persistent(W: int, S: int, P: int, t_math: float, t_la: float, t_lb: float,
                      t_epi: float, two_dma: bool = False):
    """One pipeline over W tiles of S K-iterations each (j = 1 .. W S): the
    same recurrences, with the epilogue of tile r delaying MATH of the first
    K-iteration of tile r + 1."""
    n = W * S
    Sa = [0.0] * (n + 1)
    Sb = [0.0] * (n + 1)
    Sm = [0.0] * (n + 1)
    for j in range(1, n + 1):
        if two_dma:
            Sa[j] = 0.0 if j == 1 else Sa[j - 1] + t_la
            Sb[j] = 0.0 if j == 1 else Sb[j - 1] + t_lb
            if j - P >= 1:
                Sa[j] = max(Sa[j], Sm[j - P] + t_math)
                Sb[j] = max(Sb[j], Sm[j - P] + t_math)
            ready = max(Sa[j] + t_la, Sb[j] + t_lb)
        else:
            Sa[j] = 0.0 if j == 1 else Sb[j - 1] + t_lb
            if j - P >= 1:
                Sa[j] = max(Sa[j], Sm[j - P] + t_math)
            Sb[j] = Sa[j] + t_la
            if j - P >= 1:
                Sb[j] = max(Sb[j], Sm[j - P] + t_math)
            ready = Sb[j] + t_lb
        Sm[j] = ready
        if j >= 2:
            prev_done = Sm[j - 1] + t_math
            if (j - 1) % S == 0:
                prev_done += t_epi
            Sm[j] = max(Sm[j], prev_done)
    return Sa, Sb, Sm


def rounds(M: int, N: int, tm: int, tn: int, slots: int) -> int:
    """Section 2.1: W = ceil(output tiles / number of SMs (here: workgroup slots))."""
    tiles = math.ceil(M / tm) * math.ceil(N / tn)
    return math.ceil(tiles / slots)


def stages(K: int, tk: int) -> int:
    """Section 2.1: S = ceil(K / T_K)."""
    return math.ceil(K / tk)


def overall_time(M, N, K, tm, tn, tk, P, slots, t_init, t_epi, t_math, t_la, t_lb,
                 two_dma=False, finish_math=False, schedule="per_round"):
    """Section 2.2 overall time: (S_m(S) + T_EPILOGUE) W + T_INIT, or the
    persistent-grid variant S_m(W S) + T_EPILOGUE + T_INIT."""
    W = rounds(M, N, tm, tn, slots)
    S = stages(K, tk)
    tail = t_epi + (t_math if finish_math else 0.0)
    if schedule == "persistent":
        _, _, Sm = events_persistent(W, S, P, t_math, t_la, t_lb, t_epi, two_dma)
        return Sm[W * S] + tail + t_init
    ev = events_two_dma if two_dma else events_one_dma
    _, _, Sm = ev(S, P, t_math, t_la, t_lb)
    return (Sm[S] + tail) * W + t_init


def synchronous_time(M, N, K, tm, tn, tk, slots, t_init, t_math, t_la, t_lb):
    """Section 2.1, synchronous kernel without overlap: (stage time x S) x W
    + T_INIT, with a stage = load A, load B, multiply."""
    W = rounds(M, N, tm, tn, slots)
    S = stages(K, tk)
    return ((t_la + t_lb + t_math) * S) * W + t_init


def total_wait(S: int, P: int, W: int, t_math, t_la, t_lb, two_dma=False):
    """Section 3.2, second objective: W x sum_i Wait(i), Wait(1) = S_b(1) +
    T_LOAD-B (for two DMA warps: when both first tiles have landed), Wait(i)
    = S_m(i) - (S_m(i-1) + T_MATH)."""
    ev = events_two_dma if two_dma else events_one_dma
    Sa, Sb, Sm = ev(S, P, t_math, t_la, t_lb)
    w = Sm[1]
    for i in range(2, S + 1):
        w += Sm[i] - (Sm[i - 1] + t_math)
    return W * w


def two_point_fit(work1: float, t1: float, work2: float, t2: float):
    """Section 4.2 calibration: throughput = (work' - work'') / (t' - t'')
    and startup latency = t' - work' / throughput."""
    thr = (work1 - work2) / (t1 - t2)
    return thr, t1 - work1 / thr
