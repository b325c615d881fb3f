"""The GPU resume queue's transitions on the CPU (GORIO Sec. 3.1, Fig. 1: a
ready table feeding a resume queue).

tests/queue_harness.cpp compiles the library's own transitions
(paper_2607_04415_amd/csrc/resume_queue.hpp: queue_push, queue_take,
take_fresh_lane, requeue_lane, park_begin, park_wait_on, park_withdraw,
park_recheck_wake, wake_waiters) for the host and drives them with threads
playing the executor waves and the fill waves.  Every configuration must
finish with every lane done (no stall: a lost wake leaves a lane parked for
good), no lane taken from the queue that was not QUEUED, no lane run by two
executors at once, and nothing left in the queue; the same runs again under
ThreadSanitizer.  Lane counts cross the 64-lane word of the waiter sets.  The
negative control (a parked lane that does not look at its slots again after
setting its bits) must stall: that second look is what keeps a fill that took
the waiter set first from losing the wake.  Withdrawing a resumed lane's bits
from the other slots it parked on removes the wakes that find nothing ready.
"""
import json
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
SRC = ROOT / "tests" / "queue_harness.cpp"


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    d = tmp_path_factory.mktemp("queue")
    out = {}
    for name, flags in (("plain", ["-O2"]), ("tsan", ["-O1", "-g", "-fsanitize=thread"])):
        exe = d / f"queue_harness_{name}"
        subprocess.run(["g++", *flags, "-std=c++17", "-pthread", "-Wall", "-o", str(exe), str(SRC)], check=True)
        out[name] = exe
    return out


def run(exe, lanes, executors, fillers, steps, max_waits, seed, stall_s=10, pause_us=0, withdraw=1, control=0,
        timeout=180):
    args = [lanes, executors, fillers, steps, max_waits, seed, stall_s, pause_us, withdraw, control]
    p = subprocess.run([str(exe), *map(str, args)], capture_output=True, text=True, timeout=timeout)
    assert p.returncode == 0, p.stdout + p.stderr
    assert "WARNING: ThreadSanitizer" not in p.stderr, p.stderr[-4000:]
    return json.loads(p.stdout.strip().splitlines()[-1])


CONFIGS = [
    # lanes, executors, fillers, steps, max_waits, seed, pause_us
    (40, 8, 4, 200, 4, 1, 0),
    (40, 8, 4, 200, 4, 2, 20),
    (64, 16, 8, 120, 8, 3, 0),       # one full word of waiter bits
    (65, 16, 8, 120, 8, 4, 20),      # a second word with one lane
    (130, 12, 3, 100, 3, 5, 5),
    (1, 2, 1, 500, 1, 6, 10),        # one lane, two executors
    (7, 24, 2, 300, 60, 7, 0),       # more executors than lanes, waits up to a report's cap
]


@pytest.mark.parametrize("cfg", CONFIGS, ids=[f"l{c[0]}-e{c[1]}-f{c[2]}-w{c[4]}-p{c[6]}" for c in CONFIGS])
def test_every_lane_finishes(harness, cfg):
    lanes, ex, fi, steps, waits, seed, pause = cfg
    r = run(harness["plain"], lanes, ex, fi, steps, waits, seed, pause_us=pause)
    assert not r["stalled"], r
    assert r["lanes_done"] == lanes and r["steps"] == lanes * steps, r


@pytest.mark.parametrize("cfg", [(40, 8, 4, 40, 4, 11, 0), (65, 12, 4, 30, 8, 12, 20)],
                         ids=["l40", "l65-pauses"])
def test_every_lane_finishes_under_thread_sanitizer(harness, cfg):
    lanes, ex, fi, steps, waits, seed, pause = cfg
    r = run(harness["tsan"], lanes, ex, fi, steps, waits, seed, stall_s=30, pause_us=pause, timeout=300)
    assert not r["stalled"], r
    assert r["lanes_done"] == lanes, r


def test_without_the_second_look_a_wake_is_lost(harness):
    r = run(harness["plain"], 40, 8, 4, 300, 4, 3, stall_s=1, pause_us=20, control=1)
    assert r["stalled"] and r["lanes_done"] < 40, r


def test_withdrawing_removes_wakes_that_find_nothing(harness):
    keep = run(harness["plain"], 40, 8, 4, 200, 4, 21, withdraw=0)
    gone = run(harness["plain"], 40, 8, 4, 200, 4, 21, withdraw=1)
    assert not keep["stalled"] and not gone["stalled"]
    assert keep["spurious"] > 1000, keep
    assert gone["spurious"] * 20 < keep["spurious"], (gone, keep)
