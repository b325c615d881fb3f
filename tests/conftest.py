import os
import sys
from pathlib import Path

import numpy as np
import pytest

ROOT = Path(__file__).resolve().parents[1]
if str(ROOT) not in sys.path:
    sys.path.insert(0, str(ROOT))

NO_EDGE = 0xFFFFFFFF

# a paged search that stops making progress is aborted by the library's
# watchdog well before the per-test time limit
os.environ.setdefault("GORIO_WATCHDOG_S", "90")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


@pytest.fixture(scope="session")
def orc():
    from oracle import load
    return load()


def random_graph(rng, n, R, connected=True, sentinel_frac=0.0):
    """Random out-edge lists; optionally a ring first so every node is reachable."""
    g = np.empty((n, R), np.uint32)
    for i in range(n):
        others = rng.choice(np.delete(np.arange(n), i), size=min(R, n - 1), replace=False)
        row = list(others)
        if connected and (i + 1) % n not in row:
            row[0] = (i + 1) % n
        row += [NO_EDGE] * (R - len(row))
        g[i] = row
    if sentinel_frac > 0:
        mask = rng.random((n, R)) < sentinel_frac
        if connected:
            mask[np.arange(n), [list(g[i]).index((i + 1) % n) for i in range(n)]] = False
        g[mask] = NO_EDGE
    return g


def brute_force(x, q, k, dtype="u8"):
    """Exact top-k by (squared L2, id) with numpy; float64 for float32 data."""
    if dtype == "u8":
        d = ((x.astype(np.int64) - q.astype(np.int64)[None, :]) ** 2).sum(1)
    else:
        d = ((x.astype(np.float64) - q.astype(np.float64)[None, :]) ** 2).sum(1)
    order = np.lexsort((np.arange(len(d)), d))[:k]
    return order.astype(np.uint32), d[order]


def gpu_available():
    if os.environ.get("GORIO_FORCE_NO_GPU"):
        return False
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False
