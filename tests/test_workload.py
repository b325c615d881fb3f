"""The seeded input generator: deterministic, and its graph follows the edge rule."""
import numpy as np

from workload import IndexSpec, QuerySpec, index_arrays, query_array
from workload.gen import gen_graph

SMALL = IndexSpec(n=3000, D=16, dtype="u8", clusters=4, sigma=20.0, r_near=8, r_rand=8,
                  sample=1024, seed=77)


def test_deterministic():
    a = index_arrays(SMALL, use_cache=False)
    b = index_arrays(SMALL, use_cache=False)
    for k in a:
        assert np.array_equal(a[k], b[k])
    q1 = query_array(SMALL, QuerySpec(50, 5))
    q2 = query_array(SMALL, QuerySpec(50, 5))
    assert np.array_equal(q1, q2)
    assert not np.array_equal(q1, query_array(SMALL, QuerySpec(50, 6)))


def test_edge_rule_small_clusters():
    """Clusters smaller than the sample: the near edges are the exact cluster top-R_near."""
    rng = np.random.default_rng(3)
    n, D, C = 600, 8, 3
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    labels = rng.integers(0, C, n).astype(np.uint32)
    g = gen_graph(x, labels, C, 1024, 6, 5, seed=9)
    assert g.shape == (n, 11)
    for i in range(0, n, 7):
        row = g[i].tolist()
        assert i not in row and len(set(row)) == len(row)
        same = np.flatnonzero((labels == labels[i]) & (np.arange(n) != i))
        d = ((x[same].astype(np.int64) - x[i].astype(np.int64)) ** 2).sum(1)
        want = same[np.lexsort((same, d))][:6]
        assert row[:6] == want.tolist()


def test_edge_rule_small_clusters_f32():
    """float32 vectors: the near edges are the cluster's top-R_near by float64 distance."""
    rng = np.random.default_rng(6)
    n, D, C = 500, 13, 4
    x = rng.standard_normal((n, D)).astype(np.float32)
    labels = rng.integers(0, C, n).astype(np.uint32)
    g = gen_graph(x, labels, C, 1024, 5, 3, seed=11)
    for i in range(0, n, 5):
        row = g[i].tolist()
        assert i not in row and len(set(row)) == len(row)
        same = np.flatnonzero((labels == labels[i]) & (np.arange(n) != i))
        d = ((x[same].astype(np.float64) - x[i].astype(np.float64)) ** 2).sum(1)
        want = same[np.lexsort((same, d))][:5]
        assert row[:5] == want.tolist()


def test_edge_rule_sampled_clusters():
    """Clusters larger than the sample: near edges are same-cluster and sorted by (dist, id)."""
    rng = np.random.default_rng(4)
    n, D = 4000, 8
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    labels = np.zeros(n, np.uint32)
    g = gen_graph(x, labels, 1, 256, 8, 8, seed=10)
    for i in range(0, n, 13):
        row = g[i]
        d = ((x[row[:8]].astype(np.int64) - x[i].astype(np.int64)) ** 2).sum(1)
        keys = list(zip(d.tolist(), row[:8].tolist()))
        assert keys == sorted(keys)
        assert i not in row.tolist() and len(set(row.tolist())) == 16


def test_u8_mixture_ranges():
    a = index_arrays(SMALL, use_cache=False)
    assert a["x"].dtype == np.uint8 and a["x"].shape == (3000, 16)
    assert a["graph"].dtype == np.uint32 and a["graph"].shape == (3000, 16)
    assert (a["graph"] < 3000).all()
    assert (a["centres"] >= 40).all() and (a["centres"] <= 215).all()


def test_f32_mixture_unit_norm():
    spec = IndexSpec(n=500, D=24, dtype="f32", clusters=5, sigma=0.05, r_near=4, r_rand=4, seed=5)
    a = index_arrays(spec, use_cache=False)
    assert a["x"].dtype == np.float32
    np.testing.assert_allclose(np.linalg.norm(a["x"].astype(np.float64), axis=1), 1.0, atol=1e-6)
