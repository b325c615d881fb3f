"""Host-side logic of bench.py (no GPU): the one-GPU guard and the per-leg
k-means cluster count of the paged legs."""
import subprocess
import sys
from pathlib import Path

import bench

ROOT = Path(__file__).resolve().parents[1]


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU only" in r.stderr
    assert r.stdout.strip() == ""


def test_cluster_count_by_leg_size():
    assert bench.cluster_count(-1, 10000) == 256
    assert bench.cluster_count(-1, 20000) == 256
    assert bench.cluster_count(-1, 20001) == 512
    assert bench.cluster_count(-1, 100000) == 512
    assert bench.cluster_count(0, 100000) == 0        # placement off
    assert bench.cluster_count(384, 10000) == 384     # fixed by the caller
