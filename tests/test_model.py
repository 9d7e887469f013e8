"""Performance model (Section 2) -- oracle pins and library parity (CPU only).

The oracle (oracle/model_ref.py) transcribes Eq. 1-3 and the round/overall
formulas.  It is pinned here against facts that do not reuse those formulas:
closed forms in the compute- and DMA-bound regimes, the synchronous kernel
of Section 2.1 (ring depth 1), an as-soon-as-possible schedule computed as
longest paths in the precedence graph by blind edge relaxation, the worked
wave example of Section 2.1, and the calibration fit on exact linear data.
The library's simulator (ws_model_predict / ws_model_events) must then agree
with the oracle bit for bit: both evaluate the same max-plus sums in the same
order.
"""
from __future__ import annotations

import os
import random

import pytest

from oracle import model_ref as ref

HERE = os.path.dirname(os.path.abspath(__file__))


def rnd_params(rng):
    return (rng.uniform(0.1, 5.0), rng.uniform(0.05, 3.0), rng.uniform(0.05, 3.0))


# -- pins of the oracle --------------------------------------------------------

@pytest.mark.parametrize("P", [2, 3, 4, 8])
def test_compute_bound_closed_form(P):
    t_math, t_la, t_lb = 3.0, 0.75, 1.25  # t_la + t_lb <= t_math
    _, _, Sm = ref.events_one_dma(40, P, t_math, t_la, t_lb)
    for i in range(1, 41):
        assert Sm[i] == pytest.approx(t_la + t_lb + (i - 1) * t_math, rel=1e-13)


@pytest.mark.parametrize("P", [2, 3, 5])
def test_dma_bound_closed_form(P):
    t_math, t_la, t_lb = 1.0, 0.875, 1.5  # t_la + t_lb >= t_math
    _, _, Sm = ref.events_one_dma(40, P, t_math, t_la, t_lb)
    for i in range(1, 41):
        assert Sm[i] == pytest.approx(i * (t_la + t_lb), rel=1e-13)


def test_two_dma_closed_forms():
    # compute-bound: MATH waits only for the first pair of tiles
    _, _, Sm = ref.events_two_dma(30, 2, 3.0, 1.0, 2.0)
    assert all(Sm[i] == pytest.approx(2.0 + (i - 1) * 3.0) for i in range(1, 31))
    # DMA-bound on B: MATH follows the slower DMA warp
    _, _, Sm = ref.events_two_dma(30, 2, 1.0, 0.5, 2.0)
    assert all(Sm[i] == pytest.approx(i * 2.0) for i in range(1, 31))


def test_depth_one_is_the_synchronous_kernel():
    # With one slot every load waits for the previous MATH: the overlapped
    # model must give Section 2.1's synchronous time (stage x S) x W + T_INIT.
    rng = random.Random(3)
    for _ in range(50):
        t_math, t_la, t_lb = rnd_params(rng)
        M, N, K = rng.choice([256, 512, 1024]), rng.choice([256, 768]), rng.choice([128, 1024])
        t_init = rng.uniform(0, 5)
        a = ref.overall_time(M, N, K, 128, 128, 64, 1, 84, t_init, 0.0, t_math, t_la, t_lb,
                             finish_math=True)
        b = ref.synchronous_time(M, N, K, 128, 128, 64, 84, t_init, t_math, t_la, t_lb)
        assert a == pytest.approx(b, rel=1e-12)


def asap_by_relaxation(S, P, t_math, t_la, t_lb, two_dma, rng):
    """Earliest start times of the tasks LA(i), LB(i), MM(i) as longest paths
    in their precedence graph, by relaxing the edges in random order until
    nothing changes (no recurrence is evaluated)."""
    dur = {}
    edges = []  # (u, v): v starts no earlier than u finishes
    for i in range(1, S + 1):
        dur[("A", i)], dur[("B", i)], dur[("M", i)] = t_la, t_lb, t_math
        if two_dma:
            if i > 1:
                edges += [(("A", i - 1), ("A", i)), (("B", i - 1), ("B", i))]
            edges += [(("A", i), ("M", i))]
        else:
            if i > 1:
                edges.append((("B", i - 1), ("A", i)))
            edges.append((("A", i), ("B", i)))
        edges.append((("B", i), ("M", i)))
        if i > 1:
            edges.append((("M", i - 1), ("M", i)))
        if i > P:  # the slot of K-iteration i - P must be released first
            edges += [(("M", i - P), ("A", i)), (("M", i - P), ("B", i))]
    start = {t: 0.0 for t in dur}
    changed = True
    while changed:
        changed = False
        rng.shuffle(edges)
        for u, v in edges:
            if start[u] + dur[u] > start[v]:
                start[v] = start[u] + dur[u]
                changed = True
    return start


@pytest.mark.parametrize("two_dma", [False, True])
def test_events_equal_longest_paths(two_dma):
    rng = random.Random(11 + two_dma)
    ev = ref.events_two_dma if two_dma else ref.events_one_dma
    for _ in range(40):
        S, P = rng.randint(1, 12), rng.randint(1, 5)
        t_math, t_la, t_lb = rnd_params(rng)
        Sa, Sb, Sm = ev(S, P, t_math, t_la, t_lb)
        st = asap_by_relaxation(S, P, t_math, t_la, t_lb, two_dma, rng)
        for i in range(1, S + 1):
            assert Sa[i] == pytest.approx(st[("A", i)], abs=1e-9)
            assert Sb[i] == pytest.approx(st[("B", i)], abs=1e-9)
            assert Sm[i] == pytest.approx(st[("M", i)], abs=1e-9)


def test_longest_path_pin_catches_an_index_slip():
    # A release indexed one K-iteration too late (i - P + 1) must fail the pin.
    def wrong(S, P, t_math, t_la, t_lb):
        Sa, Sb, Sm = [0.0] * (S + 1), [0.0] * (S + 1), [0.0] * (S + 1)
        for i in range(1, S + 1):
            Sa[i] = 0.0 if i == 1 else Sb[i - 1] + t_lb
            if i - P + 1 >= 1 and i > 1:
                Sa[i] = max(Sa[i], Sm[i - P + 1] + t_math)
            Sb[i] = Sa[i] + t_la
            Sm[i] = max(Sb[i] + t_lb, Sm[i - 1] + t_math if i > 1 else 0.0)
        return Sa, Sb, Sm
    rng = random.Random(5)
    Sa, Sb, Sm = wrong(8, 2, 1.0, 2.0, 2.0)
    st = asap_by_relaxation(8, 2, 1.0, 2.0, 2.0, False, rng)
    assert any(abs(Sm[i] - st[("M", i)]) > 1e-6 for i in range(1, 9))


def test_persistent_equals_longest_paths_with_epilogue():
    # The persistent schedule is the same precedence graph over W S
    # K-iterations, with the epilogue as MATH work after every S-th one.
    rng = random.Random(21)
    for two_dma in (False, True):
        for _ in range(20):
            W, S, P = rng.randint(1, 4), rng.randint(1, 6), rng.randint(1, 4)
            t_math, t_la, t_lb = rnd_params(rng)
            t_epi = rng.uniform(0, 4)
            _, _, Sm = ref.events_persistent(W, S, P, t_math, t_la, t_lb, t_epi, two_dma)
            # Longest paths with MATH of the last K-iteration of each tile
            # lasting t_math + t_epi for its successor (its slot is released
            # after t_math): model the epilogue as a task E(r) between them.
            n = W * S
            start = {}
            dur = {}
            edges = []
            for j in range(1, n + 1):
                dur[("A", j)], dur[("B", j)], dur[("M", j)] = t_la, t_lb, t_math
                if two_dma:
                    if j > 1:
                        edges += [(("A", j - 1), ("A", j)), (("B", j - 1), ("B", j))]
                    edges.append((("A", j), ("M", j)))
                else:
                    if j > 1:
                        edges.append((("B", j - 1), ("A", j)))
                    edges.append((("A", j), ("B", j)))
                edges.append((("B", j), ("M", j)))
                if j > 1:
                    if (j - 1) % S == 0:
                        dur[("E", j - 1)] = t_epi
                        edges += [(("M", j - 1), ("E", j - 1)), (("E", j - 1), ("M", j))]
                    else:
                        edges.append((("M", j - 1), ("M", j)))
                if j > P:
                    edges += [(("M", j - P), ("A", j)), (("M", j - P), ("B", j))]
            start = {t: 0.0 for t in dur}
            changed = True
            while changed:
                changed = False
                rng.shuffle(edges)
                for u, v in edges:
                    if start[u] + dur[u] > start[v]:
                        start[v] = start[u] + dur[u]
                        changed = True
            for j in range(1, n + 1):
                assert Sm[j] == pytest.approx(start[("M", j)], abs=1e-9)


def test_invariants():
    rng = random.Random(7)
    for _ in range(100):
        S, P = rng.randint(2, 30), rng.randint(1, 6)
        t_math, t_la, t_lb = rnd_params(rng)
        Sa, Sb, Sm = ref.events_one_dma(S, P, t_math, t_la, t_lb)
        for i in range(1, S + 1):
            assert Sb[i] >= Sa[i] + t_la - 1e-12
            assert Sm[i] >= Sb[i] + t_lb - 1e-12
            if i > 1:
                assert Sm[i] - Sm[i - 1] >= t_math - 1e-12
                assert Sa[i] >= Sb[i - 1] + t_lb - 1e-12
            if i > P:
                assert Sa[i] >= Sm[i - P] + t_math - 1e-12


def test_wave_example_rounds():
    # Section 2.1's example: 256 output tiles over 84 SMs take four rounds.
    kv = {}
    with open(os.path.join(HERE, "golden", "paper_wave_example.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if "=" in line:
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    tiles, sms = int(kv["tiles"]), int(kv["sms"])
    assert ref.rounds(tiles, 1, 1, 1, sms) == int(kv["waves"])
    assert ref.rounds(16 * 128, 16 * 128, 128, 128, 84) == 4  # 256 tiles of 128 x 128


def test_stage_count_and_costs():
    assert ref.stages(8192, 64) == 128 and ref.stages(100, 64) == 2
    tm, la, lb = ref.linear_costs(128, 64, 32, 1000.0, 0.5, 100.0, 0.25)
    assert tm == 128 * 64 * 32 / 1000.0 + 0.5
    assert la == 128 * 32 / 100.0 + 0.25 and lb == 32 * 64 / 100.0 + 0.25


def test_two_point_fit_recovers_a_line():
    thr, lat = ref.two_point_fit(64 * 64, 64 * 64 / 250.0 + 0.75, 128 * 128, 128 * 128 / 250.0 + 0.75)
    assert thr == pytest.approx(250.0, rel=1e-12) and lat == pytest.approx(0.75, rel=1e-12)


def test_wait_objective_regimes():
    # compute-bound: MATH waits only for the first two tiles
    assert ref.total_wait(20, 3, 4, 3.0, 0.5, 1.0) == pytest.approx(4 * 1.5)
    # DMA-bound: after the first K-iteration MATH idles (t_la + t_lb - t_math) each time
    w = ref.total_wait(20, 3, 1, 1.0, 1.0, 1.5)
    assert w == pytest.approx(2.5 + 19 * (2.5 - 1.0))


# -- library parity --------------------------------------------------------------

wsgemm = pytest.importorskip("paper_2506_11209_amd.wsgemm")


def lib_params(t_init, t_epi, ct, cl, lt, ll):
    return wsgemm.ws_model_params(t_init, t_epi, ct, cl, lt, ll)


@pytest.mark.parametrize("two_dma", [0, 1])
@pytest.mark.parametrize("persistent", [0, 1])
@pytest.mark.parametrize("finish", [0, 1])
def test_library_predict_matches_oracle(two_dma, persistent, finish):
    rng = random.Random(100 + 4 * two_dma + 2 * persistent + finish)
    opts = wsgemm.model_options(two_dma, persistent, finish)
    for _ in range(60):
        tm, tn, tk = rng.choice([32, 64, 128, 256]), rng.choice([32, 64, 128, 256]), rng.choice([32, 64, 128])
        M, N, K = tm * rng.randint(1, 40), tn * rng.randint(1, 40), tk * rng.randint(1, 60)
        P, slots = rng.randint(1, 8), rng.choice([1, 84, 256, 512])
        ct, cl = rng.uniform(1e5, 1e7), rng.uniform(0, 1)
        lt, ll = rng.uniform(1e3, 1e5), rng.uniform(0, 1)
        t_init, t_epi = rng.uniform(0, 10), rng.uniform(0, 5)
        s, r = wsgemm.ws_model_predict(M, N, K, tm, tn, tk, P, slots,
                                       lib_params(t_init, t_epi, ct, cl, lt, ll), opts)
        assert s == wsgemm.WS_OK
        t_math, t_la, t_lb = ref.linear_costs(tm, tn, tk, ct, cl, lt, ll)
        assert (r.t_math, r.t_load_a, r.t_load_b) == (t_math, t_la, t_lb)
        want = ref.overall_time(M, N, K, tm, tn, tk, P, slots, t_init, t_epi, t_math, t_la, t_lb,
                                two_dma=bool(two_dma), finish_math=bool(finish),
                                schedule="persistent" if persistent else "per_round")
        assert r.total_us == want
        assert r.rounds == ref.rounds(M, N, tm, tn, slots) and r.iters == ref.stages(K, tk)
        if not persistent:
            assert r.wait_us == pytest.approx(
                ref.total_wait(r.iters, P, r.rounds, t_math, t_la, t_lb, bool(two_dma)), rel=1e-12)


@pytest.mark.parametrize("two_dma", [0, 1])
def test_library_events_match_oracle(two_dma):
    rng = random.Random(200 + two_dma)
    for persistent in (0, 1):
        opts = wsgemm.model_options(two_dma, persistent, 0)
        for _ in range(30):
            S, W, P = rng.randint(1, 20), rng.randint(1, 4), rng.randint(1, 6)
            t_math, t_la, t_lb = rnd_params(rng)
            t_epi = rng.uniform(0, 3)
            s, sa, sb, sm = wsgemm.ws_model_events(S, W, P, t_math, t_la, t_lb, t_epi, opts)
            assert s == wsgemm.WS_OK
            if persistent:
                Sa, Sb, Sm = ref.events_persistent(W, S, P, t_math, t_la, t_lb, t_epi, bool(two_dma))
            else:
                ev = ref.events_two_dma if two_dma else ref.events_one_dma
                Sa, Sb, Sm = ev(S, P, t_math, t_la, t_lb)
            assert sa == Sa[1:] and sb == Sb[1:] and sm == Sm[1:]


def test_library_model_rejects_bad_arguments():
    p = lib_params(1, 1, 1e6, 0, 1e4, 0)
    bad = [(0, 64, 64, 64, 64, 64, 2, 84), (64, 64, 64, 0, 64, 64, 2, 84),
           (64, 64, 64, 64, 64, 64, 0, 84), (64, 64, 64, 64, 64, 64, 2, 0)]
    for args in bad:
        assert wsgemm.ws_model_predict(*args, p)[0] == wsgemm.WS_ERR_INVALID_ARG
    assert wsgemm.ws_model_predict(64, 64, 64, 64, 64, 64, 2, 84, lib_params(1, 1, 0, 0, 1e4, 0))[0] \
        == wsgemm.WS_ERR_INVALID_ARG
    assert wsgemm.ws_model_events(0, 1, 2, 1.0, 1.0, 1.0, 0.0)[0] == wsgemm.WS_ERR_INVALID_ARG


def test_library_predict_with_explicit_costs_matches_oracle():
    rng = random.Random(300)
    for two_dma in (0, 1):
        for persistent in (0, 1):
            opts = wsgemm.model_options(two_dma, persistent, 0)
            for _ in range(30):
                tm, tn, tk = 256, 128, 64
                M, N, K = tm * rng.randint(1, 40), tn * rng.randint(1, 40), tk * rng.randint(1, 60)
                P, slots = rng.randint(1, 6), rng.choice([84, 256])
                t_math, t_la, t_lb = rnd_params(rng)
                t_init, t_epi = rng.uniform(0, 10), rng.uniform(0, 5)
                s, r = wsgemm.ws_model_predict_costs(M, N, K, tm, tn, tk, P, slots, t_math, t_la, t_lb,
                                                     lib_params(t_init, t_epi, 1.0, 0.0, 1.0, 0.0), opts)
                assert s == wsgemm.WS_OK
                want = ref.overall_time(M, N, K, tm, tn, tk, P, slots, t_init, t_epi, t_math, t_la,
                                        t_lb, two_dma=bool(two_dma),
                                        schedule="persistent" if persistent else "per_round")
                assert r.total_us == want
    p = lib_params(1, 1, 1, 0, 1, 0)
    assert wsgemm.ws_model_predict_costs(64, 64, 64, 64, 64, 64, 2, 84, float("nan"), 1.0, 1.0, p)[0] \
        == wsgemm.WS_ERR_INVALID_ARG


def test_package_two_point_fit_matches_oracle():
    from paper_2506_11209_amd.model import two_point_fit
    rng = random.Random(400)
    for _ in range(50):
        w1, w2 = rng.uniform(1e3, 1e6), rng.uniform(1e3, 1e6)
        t1, t2 = rng.uniform(0.1, 10), rng.uniform(0.1, 10)
        assert two_point_fit(w1, t1, w2, t2) == ref.two_point_fit(w1, t1, w2, t2)


def test_optimizer_ranks_like_brute_force_with_the_oracle():
    # The section 3.2 optimum found by exhaustive search through the library
    # must be the argmin of the oracle's overall time over the same candidates.
    from paper_2506_11209_amd.model import Params, optimize
    params = {1: Params(6.5, 1.8, 3.1e6, 0.15, 1.0e5, 0.25), 2: Params(7.3, 1.8, 4.4e6, 0.24, 2.4e5, 0.3)}
    rng = random.Random(500)
    tiles = [(128, 128, 64), (256, 128, 64), (128, 256, 32), (64, 64, 64)]
    for _ in range(10):
        M, N, K = rng.choice([2048, 4096, 8192]), rng.choice([2048, 8192]), rng.choice([1024, 8192])
        cands = []
        for t in tiles:
            for P in (2, 3, 4):
                for split in (1, 2):
                    cands.append((t, P, 4 * split, 4, rng.choice([256, 512])))
        for objective in ("time", "wait"):
            rows = optimize(M, N, K, params, cands, objective)
            def key(c):
                t, P, np_, nc, slots = c
                p = params[np_ // nc]
                tm_, la, lb = ref.linear_costs(*t, p.compute_throughput, p.compute_latency,
                                               p.load_throughput, p.load_latency)
                total = ref.overall_time(M, N, K, *t, P, slots, p.t_init, p.t_epilogue, tm_, la, lb,
                                         two_dma=(np_ // nc == 2), schedule="persistent")
                return total
            best_time = min(key(c) for c in cands)
            if objective == "time":
                assert rows[0]["time_us"] == best_time
            assert sorted(r["time_us"] for r in rows) == sorted(key(c) for c in cands)


def test_optimizer_ranks_eight_consumer_launches_only_with_their_measured_costs(tmp_path):
    # The linear fits describe the four-consumer kernels; an eight-consumer
    # candidate is ranked with its own measured costs, and left out without.
    import json
    from paper_2506_11209_amd.model import Params, load_cost_table, optimize, table_key
    params = {1: Params(6.5, 1.8, 3.1e6, 0.15, 1.0e5, 0.25)}
    cal = {"calibrations": [{"split": 1, "load_path": "registers", "table": [
        {"tile": [256, 128, 64], "stages": 3, "t_load_a": 0.5, "t_load_b": 0.3, "t_load_ab": 0.9,
         "t_math": 1.2},
        {"tile": [256, 256, 64], "stages": 2, "consumer_waves": 8, "producer_waves": 4, "t_load_a": 0.6,
         "t_load_b": 0.6, "t_load_ab": 1.0, "t_math": 1.4}]}]}
    path = tmp_path / "calib.json"
    path.write_text(json.dumps(cal))
    table = load_cost_table(str(path))
    assert table[table_key(1, "registers", (256, 128, 64))] == (1.2, 0.9 * 256 / 384, 0.9 * 128 / 384)
    assert table[table_key(1, "registers", (256, 256, 64), 8)] == (1.4, 0.5, 0.5)
    cands = [((256, 128, 64), 3, 4, 4, 256, 1), ((256, 256, 64), 2, 4, 8, 256, 1)]
    M = N = K = 8192
    with_table = optimize(M, N, K, params, cands, "time", table=table)
    assert {(tuple(r["tile"]), r["consumer_waves"]) for r in with_table} == {((256, 128, 64), 4),
                                                                          ((256, 256, 64), 8)}
    eight = next(r for r in with_table if r["consumer_waves"] == 8)
    assert eight["costs"] == "table" and eight["split"] == 1
    # 256 x 256 tiles: 1024 tiles in 4 rounds of 128 K-iterations at t_math = 1.4 us dominate
    assert eight["time_us"] > 4 * 128 * 1.4
    without = optimize(M, N, K, params, cands, "time")
    assert [r["consumer_waves"] for r in without] == [4]
