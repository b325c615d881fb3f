"""gorio_locality_order on the CPU (host code of the library; no device).

Checked against the rule written out as a plain breadth-first walk in Python,
plus the properties that make it useful: a permutation, deterministic, and
far fewer distinct pages per adjacency list than the identity placement.
"""
from collections import deque

import numpy as np
import pytest

import paper_2607_04415_amd as g
from conftest import NO_EDGE, random_graph


@pytest.fixture(scope="module", autouse=True)
def built():
    if not g.LIB_PATH.exists():
        from paper_2607_04415_amd import _build
        _build.build()


def reference_order(graph, entry, rpp):
    n, R = graph.shape
    slot = [None] * n
    nxt = 0
    seen = [False] * n
    q = deque([entry])
    seen[entry] = True
    while q:
        u = q.popleft()
        if slot[u] is None:
            slot[u] = nxt; nxt += 1
            for v in graph[u]:
                if nxt % rpp == 0:
                    break
                if v != NO_EDGE and slot[v] is None:
                    slot[v] = nxt; nxt += 1
        for v in graph[u]:
            if v != NO_EDGE and not seen[v]:
                seen[v] = True
                q.append(int(v))
    for v in range(n):
        if slot[v] is None:
            slot[v] = nxt; nxt += 1
    return np.array(slot, np.uint32)


@pytest.mark.parametrize("n,R,rpp,frac", [(300, 6, 10, 0.0), (500, 12, 3, 0.3), (64, 4, 1, 0.5), (257, 8, 64, 0.1)])
def test_matches_the_rule(n, R, rpp, frac):
    rng = np.random.default_rng(n + R)
    graph = random_graph(rng, n, R, connected=frac == 0.0, sentinel_frac=frac)
    for entry in (0, n // 2):
        got = g.locality_order(graph, entry, rpp)
        assert np.array_equal(got, reference_order(graph, entry, rpp))
        assert np.array_equal(np.sort(got), np.arange(n, dtype=np.uint32))
        assert got[entry] == 0


def test_unreachable_nodes_follow_in_id_order():
    graph = np.full((10, 2), NO_EDGE, np.uint32)
    graph[0] = [1, 2]
    got = g.locality_order(graph, 0, 4)
    assert got[:3].tolist() == [0, 1, 2]
    assert got[3:].tolist() == list(range(3, 10))


def test_neighbours_share_pages():
    """Near-neighbour graphs: adjacency lists span far fewer pages."""
    rng = np.random.default_rng(7)
    n, R, rpp = 4000, 8, 10
    pts = rng.random((n, 2))
    d = ((pts[:, None, :] - pts[None, :, :]) ** 2).sum(-1)
    np.fill_diagonal(d, np.inf)
    graph = np.argsort(d, axis=1)[:, :R].astype(np.uint32)
    perm = g.locality_order(graph, 0, rpp)

    def pages_per_row(slot):
        return np.mean([len({int(slot[v]) // rpp for v in graph[u]}) for u in range(n)])
    assert pages_per_row(perm) < 0.6 * pages_per_row(np.arange(n))


def test_rejects():
    graph = np.zeros((5, 2), np.uint32)
    for args in ((graph, 5, 10), (graph, 0, 0)):
        with pytest.raises(g.GorioError) as e:
            g.locality_order(*args)
        assert e.value.status == g.EINVAL
    bad = graph.copy(); bad[1, 1] = 7
    with pytest.raises(g.GorioError):
        g.locality_order(bad, 0, 4)
