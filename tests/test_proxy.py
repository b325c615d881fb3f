"""The transport proxy on the CPU, with host threads playing the GPU side.

Exactly-once completion, the injected latency honoured, the outstanding cap
respected, completions reordered under jitter; once more under
ThreadSanitizer and AddressSanitizer.
"""
import json
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
SRC = [ROOT / "tests" / "proxy_harness.cpp", ROOT / "paper_2607_04415_amd" / "csrc" / "proxy.cpp"]


def build(tmp_path, sanitize=None):
    exe = tmp_path / f"harness_{sanitize or 'plain'}"
    cmd = ["g++", "-O2", "-std=c++17", "-pthread", "-o", str(exe), *map(str, SRC)]
    if sanitize:
        cmd[1:1] = [f"-fsanitize={sanitize}", "-g"]
    subprocess.run(cmd, check=True)
    return exe


def run(exe, *args, timeout=120):
    out = subprocess.run([str(exe), *map(str, args)], capture_output=True, text=True, timeout=timeout)
    assert out.returncode == 0, out.stdout + out.stderr
    return json.loads(out.stdout.strip().splitlines()[-1])


@pytest.mark.parametrize("latency,cap,rings", [(0.0, 4096, 1), (20.0, 4096, 1), (50.0, 64, 1),
                                               (0.0, 4096, 16), (20.0, 4096, 7)])
def test_proxy_exactly_once_latency_cap(tmp_path, latency, cap, rings):
    exe = build(tmp_path)
    r = run(exe, 100000, latency, cap, 10000, 4, rings)
    assert r["missing"] == 0 and r["duplicated"] == 0 and r["early"] == 0 and r["bad"] == 0
    assert r["max_in_flight"] <= cap


def test_proxy_jitter_reorders_and_stays_exactly_once(tmp_path):
    exe = build(tmp_path)
    r = run(exe, 50000, 10.0, 4096, 10000, 4, 4, 200.0)
    assert r["missing"] == 0 and r["duplicated"] == 0 and r["early"] == 0 and r["bad"] == 0
    assert r["reordered"] > 0, "jitter did not reorder any completion"
    r0 = run(exe, 50000, 10.0, 4096, 10000, 4, 1, 0.0)
    assert r0["missing"] == 0 and r0["duplicated"] == 0


def test_proxy_under_address_sanitizer(tmp_path):
    exe = build(tmp_path, sanitize="address")
    r = run(exe, 20000, 5.0, 1024, 2000, 3, 4, 20.0, timeout=300)
    assert r["missing"] == 0 and r["duplicated"] == 0


def test_proxy_under_thread_sanitizer(tmp_path):
    exe = build(tmp_path, sanitize="thread")
    r = run(exe, 20000, 5.0, 1024, 2000, 3, 4, timeout=300)
    assert r["missing"] == 0 and r["duplicated"] == 0
