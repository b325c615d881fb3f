"""The page cache's slot state machine on the CPU (GORIO Sec. 3.2).

tests/slot_harness.cpp compiles the library's own slot transitions
(paper_2607_04415_amd/csrc/slot_state.hpp: acquire_page, claim_slot, unpin,
slot_ready, mark_ready) for the host and drives them with threads playing the
query waves and the fill side. Every configuration must finish with every
access completed, no page read through a slot that held another page, no pin
left, no slot left LOADING, a consistent page-to-slot map and no descriptor
left; the same runs once more under ThreadSanitizer. Two negative controls
(a read after the unpin; READY published before the page bytes) show that
the read check catches the mistakes it is there for.  Runs with pauses at the
state machine's pause points (GORIO_SLOT_PAUSE) widen its races; one of them
is the regression test of a stale lookup joining a slot that was given back.

The first two configurations are the paged search's smallest tested cache:
128 slots (two query slots per wave, float32 rows of 96 dimensions with R=8,
9 records per page), where the library runs at most slots / (2 x 32) = 2
queries at once, with up to 32 requests each.
"""
import json
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
SRC = ROOT / "tests" / "slot_harness.cpp"


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    d = tmp_path_factory.mktemp("slot")
    out = {}
    for name, flags in (("plain", ["-O2"]), ("tsan", ["-O1", "-g", "-fsanitize=thread"])):
        exe = d / f"slot_harness_{name}"
        subprocess.run(["g++", *flags, "-std=c++17", "-pthread", "-Wall", "-o", str(exe), str(SRC)], check=True)
        out[name] = exe
    return out


def run(exe, slots, pages, live, pending, queries, accesses, fillers, latency_us, seed, control=0,
        stall_s=10, timeout=120, pause_us=0):
    args = [slots, pages, live, pending, queries, accesses, fillers, latency_us, seed, stall_s, control, pause_us]
    p = subprocess.run([str(exe), *map(str, args)], capture_output=True, text=True, timeout=timeout)
    assert p.returncode == 0, p.stdout + p.stderr
    # ThreadSanitizer reports on stderr and keeps going; any report fails
    assert "WARNING: ThreadSanitizer" not in p.stderr, p.stderr[-4000:]
    r = json.loads(p.stdout.strip().splitlines()[-1])
    r["expected_accesses"] = queries * accesses
    return r


def assert_clean(r):
    assert not r["stalled"], r
    assert r["queries"] > 0 and r["completed_accesses"] == r["expected_accesses"], r
    assert r["bad_reads"] == 0, r
    assert r["pins_left"] == 0 and r["loading_left"] == 0, r
    assert r["unmapped_ready"] == 0 and r["map_errors"] == 0, r
    assert r["descriptors_left"] == 0 and r["served"] == r["misses"], r


CONFIGS = {
    # slots, pages, queries in flight, max pending, queries, accesses, fillers, latency (us)
    "128-slots-2x32-l0": (128, 2000, 2, 32, 200, 300, 2, 0.0),
    "128-slots-2x32-l20": (128, 2000, 2, 32, 100, 300, 2, 20.0),
    "64-slots-pins-oversubscribed": (64, 4000, 8, 16, 400, 200, 3, 5.0),
    "8-slots": (8, 64, 4, 4, 1000, 100, 2, 0.0),
    "all-pages-fit": (16, 16, 8, 8, 1000, 100, 2, 0.0),
    "10000-slots-30x32": (10000, 100000, 30, 32, 300, 2000, 4, 0.0),
}


@pytest.mark.parametrize("name", list(CONFIGS))
def test_slot_state_machine(harness, name):
    r = run(harness["plain"], *CONFIGS[name], seed=list(CONFIGS).index(name) + 1)
    assert_clean(r)
    assert r["misses"] > 0 and r["hits"] > 0


@pytest.mark.parametrize("seed", [9, 10, 11, 12])
def test_stale_lookup_never_joins_a_slot_given_back(harness, seed):
    """A lookup that read a page's slot, then paused while the slot was
    evicted, claimed again for the same page by a wave that lost the race to
    map it and was given back unfilled, must not wait on that slot: it joins a
    LOADING slot only while the page maps to it.  Threads pause at the state
    machine's pause points (after a lookup, after a claim, before a give-back)
    to make that interleaving common; without the check every run of this
    configuration left queries waiting on EMPTY slots for good."""
    r = run(harness["plain"], 8, 24, 6, 4, 2000, 100, 2, 0.0, seed=seed, stall_s=5, pause_us=100)
    assert_clean(r)


@pytest.mark.parametrize("cfg", [(2, 10, 2, 1, 400, 50, 1), (4, 40, 3, 2, 400, 100, 2), (32, 200, 12, 4, 200, 100, 3)],
                         ids=["2-slots-1-request", "4-slots", "32-slots-12-queries"])
def test_slot_state_machine_with_pauses(harness, cfg):
    slots, pages, live, pending, queries, accesses, fillers = cfg
    r = run(harness["plain"], slots, pages, live, pending, queries, accesses, fillers, 0.0, seed=21, pause_us=50)
    assert_clean(r)


@pytest.mark.parametrize("name", ["128-slots-2x32-l20", "8-slots"])
def test_slot_state_machine_tsan(harness, name):
    slots, pages, live, pending, queries, accesses, fillers, lat = CONFIGS[name]
    r = run(harness["tsan"], slots, pages, live, pending, min(queries, 200), accesses, fillers, lat, seed=9)
    assert_clean(r)


def test_slot_state_machine_tsan_with_pauses(harness):
    r = run(harness["tsan"], 8, 24, 6, 4, 300, 100, 2, 0.0, seed=13, pause_us=100)
    assert_clean(r)


@pytest.mark.parametrize("control", [1, 2], ids=["read-after-unpin", "ready-before-bytes"])
def test_negative_controls_are_caught(harness, control):
    r = run(harness["plain"], 8, 64, 4, 4, 500, 100, 2, 0.0, seed=3, control=control)
    assert r["bad_reads"] > 0, r
