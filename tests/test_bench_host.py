"""Host-side logic of bench.py (no GPU): the one-GPU guard, the k-means
cluster count of the paged legs, and the roofline and baseline helpers."""
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


def test_cluster_count_default_and_overrides():
    assert bench.cluster_count(-1, 10000) == 512
    assert bench.cluster_count(-1, 100000) == 512
    assert bench.cluster_count(0, 100000) == 0        # placement off
    assert bench.cluster_count(384, 10000) == 384     # fixed by the caller


def test_algorithmic_bytes_sources():
    st = {"expansions": 10, "evaluations": 100, "reevaluations": 7}
    # oracle counts when given, the GPU's lower bound (evaluations minus unrecorded) otherwise
    assert bench.algorithmic_bytes(st, 64, 128, oracle_evals=95) == (10 * 260 + 95 * 128, "oracle")
    b, src = bench.algorithmic_bytes(st, 64, 384)
    assert b == 10 * 260 + 93 * 384 and src.startswith("gpu lower bound")


def test_roofline_of_reports_both_rates():
    class W:
        class index:
            vec_bytes = 384
    res = {"stats": {"expansions": 1000, "evaluations": 20000, "reevaluations": 500},
           "kernel_ms": [2.0, 2.0]}
    r = bench.roofline_of(res, W, 64, None, 9.0e9, "k")
    alg = 1000 * 260 + 19500 * 384
    assert r["algorithmic_bytes_per_launch"] == alg
    assert abs(r["achieved"] - alg / 2e-3 / 1e9) < 0.1
    assert abs(r["algorithmic_upper_gbs"] - (1000 * 260 + 20000 * 384) / 2e-3 / 1e9) < 0.1
    assert r["traffic_gbs"] == round(9.0e9 / 2e-3 / 1e9, 1)
    assert r["frac"] == round(r["achieved"] / bench.HBM_PEAK_GBS, 4)


def test_oracle_threads_capped_by_the_cpu_share(monkeypatch):
    monkeypatch.setenv("OMP_NUM_THREADS", "3")
    t, nproc = bench.oracle_threads()
    assert t == min(3, nproc) and nproc >= 1
