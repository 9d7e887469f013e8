"""Host model of the circular-buffer protocol (tests/ring_protocol_model.cpp),
built with g++ and ThreadSanitizer, over the ring arithmetic the kernels use
(paper_2506_11209_amd/csrc/ws_ring.hpp).

The correct protocol must run every configuration without a data race, a
wrong tag or a timeout; each planted mistake must be caught: a slot released
before it is read or read one signal early races (ThreadSanitizer) and
returns wrong tags, a producer that skips its wait on a counter value read
from the wrong slot races, and a dropped signal ends in the watchdog's
timeout instead of a hang.

The deferred-signal mode (the LDS-DMA producer, which signals a K-iteration
only once later ones are in flight, against consumers that check K-iteration
q + 1 full before releasing q) must run for every signal lag, and a producer
that drains one K-iteration too few before blocking must end in the
watchdog's timeout."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCE = os.path.join(ROOT, "tests", "ring_protocol_model.cpp")
INCLUDE = os.path.join(ROOT, "paper_2506_11209_amd", "csrc")

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")

TSAN_RACE_STATUS = 66  # ThreadSanitizer's exit status when it reported a race


@pytest.fixture(scope="module")
def models(tmp_path_factory):
    out = tmp_path_factory.mktemp("ring_model")
    built = {}
    for plant in ("", "PLANT_EARLY_RELEASE", "PLANT_EARLY_READ", "PLANT_DROP_SIGNAL", "PLANT_SHORT_DRAIN",
                  "PLANT_PEEK_WRONG_SLOT"):
        exe = str(out / ("model_" + (plant or "ok")))
        cmd = ["g++", "-std=c++17", "-O1", "-g", "-pthread", "-fsanitize=thread", "-I" + INCLUDE, SOURCE,
               "-o", exe]
        if plant:
            cmd.insert(1, "-D" + plant)
        subprocess.run(cmd, check=True)
        built[plant] = exe
    return built


def run(exe, P, NP, NC, T, limit_ms=5000, lag=None):
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=0")
    args = [exe, str(P), str(NP), str(NC), str(T), str(limit_ms)] + ([] if lag is None else [str(lag)])
    r = subprocess.run(args, capture_output=True, text=True, timeout=120, env=env)
    return r.returncode, r.stdout + r.stderr


# ring depths, producer / consumer wave counts of the kernel's arrangements
# (1:1 and 2:1 with one or four consumer waves), and K-iteration counts well
# beyond the ring depth
CONFIGS = [(P, NP, NC, T) for (NP, NC) in ((1, 1), (2, 1), (4, 4), (8, 4)) for P in (1, 2, 3, 8)
           for T in (1, 7, 1500)]


@pytest.mark.parametrize("P,NP,NC,T", CONFIGS)
def test_protocol_is_race_free_and_delivers_every_tile(models, P, NP, NC, T):
    rc, out = run(models[""], P, NP, NC, T)
    assert rc == 0, out
    assert "ThreadSanitizer" not in out, out


@pytest.mark.parametrize("P,NP,NC", [(2, 4, 4), (3, 8, 4), (1, 1, 1)])
def test_early_release_is_caught(models, P, NP, NC):
    rc, out = run(models["PLANT_EARLY_RELEASE"], P, NP, NC, 2000)
    assert rc == TSAN_RACE_STATUS and "data race" in out, out


@pytest.mark.parametrize("P,NP,NC", [(2, 4, 4), (3, 8, 4), (1, 1, 1)])
def test_early_read_is_caught(models, P, NP, NC):
    rc, out = run(models["PLANT_EARLY_READ"], P, NP, NC, 2000)
    assert rc == TSAN_RACE_STATUS and "data race" in out, out


@pytest.mark.parametrize("P,NP,NC", [(2, 4, 4), (3, 8, 4), (1, 1, 1)])
def test_dropped_signal_times_out_instead_of_hanging(models, P, NP, NC):
    rc, out = run(models["PLANT_DROP_SIGNAL"], P, NP, NC, 2000, limit_ms=300)
    assert rc == 2, out
    assert "ThreadSanitizer" not in out, out


@pytest.mark.parametrize("P,NP,NC", [(2, 4, 4), (3, 8, 4), (4, 4, 8)])
def test_reading_the_wrong_slot_with_the_signal_is_caught(models, P, NP, NC):
    # the signalled slot's counter says nothing about the next slot's
    # previous use: the producer overwrites it while consumers still read it
    rc, out = run(models["PLANT_PEEK_WRONG_SLOT"], P, NP, NC, 2000)
    assert rc == TSAN_RACE_STATUS and "data race" in out, out


# the LDS-DMA producer's lags: 1 for two slots, P - 2 beyond; 0 and larger
# lags exercise the drain before a blocking wait
DEFERRED = [(P, NP, NC, lag) for (NP, NC) in ((1, 1), (4, 4), (4, 8), (8, 4)) for P in (2, 3, 4, 8)
            for lag in sorted({0, 1, max(P - 2, 0), P - 1, P + 3})]


@pytest.mark.parametrize("P,NP,NC,lag", DEFERRED)
def test_deferred_signals_keep_the_ring_live(models, P, NP, NC, lag):
    rc, out = run(models[""], P, NP, NC, 1500, lag=lag)
    assert rc == 0, out
    assert "ThreadSanitizer" not in out, out


@pytest.mark.parametrize("P,NP,NC", [(2, 4, 4), (4, 4, 8), (3, 1, 1)])
def test_short_drain_times_out(models, P, NP, NC):
    # with a lag of P - 1 or more a blocked producer still holds K-iteration
    # q - P + 1, which the consumers need before they release q - P
    rc, out = run(models["PLANT_SHORT_DRAIN"], P, NP, NC, 2000, limit_ms=300, lag=P + 3)
    assert rc == 2, out
    assert "ThreadSanitizer" not in out, out


def test_deferred_mode_rejects_one_slot(models):
    rc, _ = run(models[""], 1, 1, 1, 10, lag=0)
    assert rc == 3
