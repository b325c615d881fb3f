"""Pins for the CPU oracle: it is checked against things other than itself.

* hand-worked traces (tests/golden/trace8.json, derivation in trace8.md);
* closed forms (distance, medoid) computed with numpy in a different way;
* special cases that reduce to exact k-NN (complete graph; L >= n on a
  connected graph), checked against numpy brute force;
* W = 1 reduces to DiskANN's GreedySearch (Subramanya et al., NeurIPS 2019,
  Algorithm 1), written here with Python sets from that textbook statement;
* invariants (V monotone, F strictly sorted, F == top-L(V)) via debug mode;
* invariance to adjacency order, node placement and record/page padding.
"""
import json
import math
from pathlib import Path

import numpy as np
import pytest

from conftest import NO_EDGE, brute_force, random_graph

GOLDEN = Path(__file__).parent / "golden"


# --------------------------------------------------------------------------- #
# hand-worked traces
# --------------------------------------------------------------------------- #
def _trace8():
    t = json.loads((GOLDEN / "trace8.json").read_text())
    x = np.array(t["vectors"], np.uint8)
    g = np.array(t["graph"], np.uint32)
    return t, x, g


def test_trace8_medoid(orc):
    t, x, _ = _trace8()
    assert orc.medoid(x) == t["medoid"]["entry"]


@pytest.mark.parametrize("case", range(8))
def test_trace8_search(orc, case):
    t, x, g = _trace8()
    c = t["cases"][case]
    ix = orc.pack(x, g)
    ids, dists, counts, trace = ix.search(np.array(c["query"], np.uint8), c["k"], c["L"], c["W"],
                                          entry=t["medoid"]["entry"], debug=True, trace_cap=8)
    assert ids[0].tolist() == c["ids"]
    assert dists[0].tolist() == c["dists"]
    assert int(counts[0]["evaluations"]) == c["evaluations"]
    assert int(counts[0]["expansions"]) == c["expansions"]
    assert int(counts[0]["iterations"]) == c["iterations"]
    n_exp = c["expansions"]
    assert trace[0][:n_exp].tolist() == c["expanded_order"]


# --------------------------------------------------------------------------- #
# closed forms
# --------------------------------------------------------------------------- #
def test_distance_u8_closed_form(orc):
    rng = np.random.default_rng(5)
    for D in (1, 4, 7, 128, 200):
        for _ in range(20):
            a = rng.integers(0, 256, D, dtype=np.uint8)
            b = rng.integers(0, 256, D, dtype=np.uint8)
            want = int(np.dot(a.astype(np.int64) - b, a.astype(np.int64) - b))
            assert orc.dist(a, b) == want
    a = np.zeros(128, np.uint8)
    b = np.full(128, 255, np.uint8)
    assert orc.dist(a, b) == 128 * 255 * 255 == 8_323_200
    assert orc.dist(b, a) == 8_323_200
    assert orc.dist(a, a) == 0


def test_distance_f32_error_bound(orc):
    """Sequential float32 sum of squares against the exact value.

    Each term fl(fl(a-b)^2) carries relative error <= gamma_2 and recursive
    summation of D non-negative terms adds gamma_{D-1} (Higham, Accuracy and
    Stability, Sec. 4.2), so |computed - exact| <= gamma_{D+2} * exact.
    """
    rng = np.random.default_rng(6)
    u = 2.0 ** -24
    for D in (1, 3, 96, 128, 300):
        g = (D + 2) * u / (1 - (D + 2) * u)
        for _ in range(30):
            a = rng.standard_normal(D).astype(np.float32)
            b = rng.standard_normal(D).astype(np.float32)
            exact = math.fsum(float(np.float64(x) - np.float64(y)) ** 2 for x, y in zip(a, b))
            got = float(orc.dist(a, b))
            assert abs(got - exact) <= g * exact + 1e-45
    z = np.zeros(96, np.float32)
    assert float(orc.dist(z, z)) == 0.0


def test_distance_f32_sequential_recipe(orc):
    """The float32 recipe is the plain left-to-right loop with no fused multiply-add.

    Documents the exact rounding sequence; the error-bound test above is the pin.
    """
    rng = np.random.default_rng(7)
    for _ in range(50):
        a = (rng.standard_normal(96) * 3).astype(np.float32)
        b = (rng.standard_normal(96) * 3).astype(np.float32)
        acc = np.float32(0)
        for x, y in zip(a, b):
            t = np.float32(x - y)
            acc = np.float32(acc + np.float32(t * t))
        assert orc.dist(a, b).view(np.uint32) == acc.view(np.uint32)


def test_medoid_u8_closed_form(orc):
    rng = np.random.default_rng(8)
    for n, D in ((1, 4), (2, 1), (50, 16), (999, 128)):
        x = rng.integers(0, 256, (n, D), dtype=np.uint8)
        s = x.astype(np.int64).sum(0)
        c = (s + n // 2) // n
        d = ((x.astype(np.int64) - c[None, :]) ** 2).sum(1)
        want = int(np.flatnonzero(d == d.min())[0])
        assert orc.medoid(x) == want
    # rounding matters: x = {0, 1}, n = 2 -> c = floor((1 + 1) / 2) = 1 -> node 1
    assert orc.medoid(np.array([[0], [1]], np.uint8)) == 1
    # ties go to the smaller id
    assert orc.medoid(np.array([[5, 5], [5, 5], [0, 0], [10, 10]], np.uint8)) == 0


def test_medoid_f32_closed_form(orc):
    rng = np.random.default_rng(9)
    for n, D in ((1, 3), (40, 8), (500, 96)):
        x = rng.standard_normal((n, D)).astype(np.float32)
        c = (np.add.accumulate(x.astype(np.float64), axis=0)[-1] / n).astype(np.float32)
        exact = ((x.astype(np.float64) - c.astype(np.float64)[None, :]) ** 2).sum(1)
        got = orc.medoid(x)
        # the chosen node is the minimiser up to float32 rounding of the distance
        assert exact[got] <= exact.min() * (1 + 4 * D * 2.0 ** -24)


# --------------------------------------------------------------------------- #
# packing: an independent numpy decoder reads the oracle's pages
# --------------------------------------------------------------------------- #
def _decode(pages, n, D, R, vec_dtype, rec_bytes, rpp, page_bytes=4096, node_to_slot=None,
            vectors_first=False):
    """Reads the layout as the header documents it: contiguous records, or the
    page's vectors (each padded to a multiple of 16 bytes) followed by its
    adjacency blocks."""
    vb = D * np.dtype(vec_dtype).itemsize
    V = -(-vb // 16) * 16
    xs = np.empty((n, D), vec_dtype)
    deg = np.empty(n, np.uint32)
    ids = np.empty((n, R), np.uint32)
    for v in range(n):
        s = v if node_to_slot is None else int(node_to_slot[v])
        page, i = (s // rpp) * page_bytes, s % rpp
        if vectors_first:
            vec_at = page + i * V
            adj_at = page + rpp * V + i * (rec_bytes - V)
        else:
            vec_at = page + i * rec_bytes
            adj_at = vec_at + vb
        xs[v] = pages[vec_at:vec_at + vb].view(vec_dtype)
        deg[v] = pages[adj_at:adj_at + 4].view("<u4")[0]
        ids[v] = pages[adj_at + 4:adj_at + 4 + 4 * R].view("<u4")
    return xs, deg, ids


@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_pack_roundtrip(orc, dtype):
    rng = np.random.default_rng(10)
    n, D, R = 137, 12, 6
    x = (rng.integers(0, 256, (n, D), dtype=np.uint8) if dtype == "u8"
         else rng.standard_normal((n, D)).astype(np.float32))
    g = random_graph(rng, n, R, sentinel_frac=0.3)
    perm = rng.permutation(n).astype(np.uint32)
    for node_to_slot in (None, perm):
        for vf in (False, True):
            ix = orc.pack(x, g, node_to_slot=node_to_slot, vectors_first=vf)
            vb = D * x.dtype.itemsize
            assert ix.record_bytes == (-(-vb // 16) * 16 if vf else vb) + 4 + 4 * R
            xs, deg, ids = _decode(ix.pages, n, D, R, x.dtype, ix.record_bytes, ix.rpp,
                                   node_to_slot=node_to_slot, vectors_first=vf)
            assert np.array_equal(xs, x)
            for v in range(n):
                real = [e for e in g[v] if e != NO_EDGE]
                assert deg[v] == len(real)
                assert ids[v].tolist() == real + [NO_EDGE] * (R - len(real))
            # unused page tail is zero
            used = ix.rpp * ix.record_bytes
            pg = ix.pages.reshape(-1, 4096)
            assert not pg[:, used:].any()


def test_pack_rejects(orc):
    rng = np.random.default_rng(11)
    x = rng.integers(0, 256, (20, 8), dtype=np.uint8)
    g = random_graph(rng, 20, 4)
    bad = g.copy(); bad[3, 1] = 20                     # id >= n that is not "no edge"
    with pytest.raises(ValueError):
        orc.pack(x, bad)
    with pytest.raises(ValueError):                    # record larger than declared
        orc.pack(x, g, record_bytes=10)
    with pytest.raises(ValueError):                    # records overflow the page
        orc.pack(x, g, record_bytes=40, records_per_page=200)
    with pytest.raises(ValueError):                    # not a permutation
        orc.pack(x, g, node_to_slot=np.zeros(20, np.uint32))
    with pytest.raises(ValueError):                    # vectors first: 16 + 4 + 16 bytes needed
        orc.pack(x, g, record_bytes=28, vectors_first=True)


# --------------------------------------------------------------------------- #
# exact special cases
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_complete_graph_is_exact(orc, dtype):
    rng = np.random.default_rng(12)
    n, D = 150, 16
    x = (rng.integers(0, 256, (n, D), dtype=np.uint8) if dtype == "u8"
         else rng.standard_normal((n, D)).astype(np.float32))
    g = np.array([[j for j in range(n) if j != i] for i in range(n)], np.uint32)
    ix = orc.pack(x, g)
    qs = (rng.integers(0, 256, (20, D), dtype=np.uint8) if dtype == "u8"
          else rng.standard_normal((20, D)).astype(np.float32))
    entry = orc.medoid(x)
    for k, L, W in ((1, 1, 1), (10, 10, 1), (10, 32, 4), (5, 64, 8)):
        ids, dists, _, _ = ix.search(qs, k, L, W, entry, debug=True)
        for qi in range(len(qs)):
            want_ids, want_d = brute_force(x, qs[qi], k, dtype)
            assert ids[qi].tolist() == want_ids.tolist()
            if dtype == "u8":
                assert dists[qi].tolist() == want_d.tolist()
            else:
                np.testing.assert_allclose(dists[qi], want_d, rtol=1e-5)


@pytest.mark.parametrize("W", [1, 2, 4, 8])
def test_L_ge_n_is_exact(orc, W):
    rng = np.random.default_rng(13 + W)
    n, D, R = 96, 8, 4
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    g = random_graph(rng, n, R, connected=True, sentinel_frac=0.2)
    ix = orc.pack(x, g)
    qs = rng.integers(0, 256, (25, D), dtype=np.uint8)
    for entry in (0, 17, orc.medoid(x)):
        ids, dists, counts, _ = ix.search(qs, 10, n, W, entry, debug=True)
        assert (counts["evaluations"] == n).all()      # whole reachable set
        assert (counts["expansions"] == n).all()
        for qi in range(len(qs)):
            want_ids, want_d = brute_force(x, qs[qi], 10)
            assert ids[qi].tolist() == want_ids.tolist()
            assert dists[qi].tolist() == want_d.tolist()


def test_ties_break_by_id(orc):
    # groups of identical vectors -> equal distances; smaller ids first
    base = np.array([[0, 0], [10, 10], [20, 20]], np.uint8)
    x = np.repeat(base, 4, axis=0)[[3, 7, 11, 0, 4, 8, 1, 5, 9, 2, 6, 10]]
    n = len(x)
    # descending adjacency: insertion order is the reverse of id order
    g = np.array([[j for j in reversed(range(n)) if j != i] for i in range(n)], np.uint32)
    ix = orc.pack(x, g)
    ids, dists, _, _ = ix.search(np.array([1, 1], np.uint8), 8, 12, 2, entry=5)
    d = ((x.astype(int) - 1) ** 2).sum(1)
    order = sorted(range(n), key=lambda v: (d[v], v))[:8]
    assert ids[0].tolist() == order
    assert dists[0].tolist() == [int(d[v]) for v in order]


def test_unreachable_pads(orc):
    # two components; entry in the small one
    x = np.arange(10, dtype=np.uint8).reshape(10, 1) * 10
    g = np.full((10, 2), NO_EDGE, np.uint32)
    g[0] = [1, NO_EDGE]; g[1] = [2, 0]; g[2] = [0, NO_EDGE]
    for i in range(3, 10):
        g[i] = [3 + (i - 2) % 7, NO_EDGE]
    ix = orc.pack(x, g)
    ids, dists, counts, _ = ix.search(np.array([95], np.uint8), 5, 8, 2, entry=0)
    assert ids[0].tolist()[:3] == [2, 1, 0]
    assert ids[0].tolist()[3:] == [NO_EDGE, NO_EDGE]
    assert dists[0].tolist()[3:] == [2 ** 31 - 1] * 2
    assert counts[0]["evaluations"] == 3
    xf = x.astype(np.float32)
    ixf = orc.pack(xf, g)
    _, df, _, _ = ixf.search(np.array([95.0], np.float32), 5, 8, 2, entry=0)
    assert np.isinf(df[0][3:]).all()


# --------------------------------------------------------------------------- #
# W = 1: DiskANN GreedySearch, from its textbook statement
# --------------------------------------------------------------------------- #
def diskann_greedy(x, g, q, entry, k, Lsize):
    """Algorithm 1 of Subramanya et al. (2019) with ties broken by id.

    Lset <- {s}; Vis <- {}; while Lset \\ Vis nonempty: p* <- closest in Lset \\ Vis;
    Lset <- Lset u N_out(p*); Vis <- Vis u {p*}; keep the Lsize closest of Lset.
    """
    def key(v):
        return (int(((x[v].astype(np.int64) - q.astype(np.int64)) ** 2).sum()), v)
    Lset = {entry}
    Vis = set()
    seen = {entry}
    order = []
    while Lset - Vis:
        p = min(Lset - Vis, key=key)
        nb = {int(v) for v in g[p] if v != NO_EDGE}
        Lset |= nb
        seen |= nb
        Vis.add(p)
        order.append(p)
        if len(Lset) > Lsize:
            Lset = set(sorted(Lset, key=key)[:Lsize])
    best = sorted(Lset, key=key)[:k]
    return best, [key(v)[0] for v in best], order, len(seen)


def test_W1_is_diskann_greedy_search(orc):
    rng = np.random.default_rng(14)
    for trial in range(6):
        n, D, R = 300, 8, 6
        x = rng.integers(0, 256, (n, D), dtype=np.uint8)
        g = random_graph(rng, n, R, connected=trial % 2 == 0, sentinel_frac=0.1 * (trial % 3))
        ix = orc.pack(x, g)
        entry = orc.medoid(x)
        qs = rng.integers(0, 256, (10, D), dtype=np.uint8)
        for L in (1, 5, 16, 40):
            k = min(L, 5)
            ids, dists, counts, trace = ix.search(qs, k, L, 1, entry, trace_cap=n)
            for qi in range(len(qs)):
                best, bd, order, nseen = diskann_greedy(x, g, qs[qi], entry, k, L)
                assert ids[qi].tolist()[:len(best)] == best
                assert dists[qi].tolist()[:len(best)] == bd
                assert trace[qi][:len(order)].tolist() == order
                assert int(counts[qi]["expansions"]) == len(order)
                assert int(counts[qi]["evaluations"]) == nseen


# --------------------------------------------------------------------------- #
# invariants and invariances
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_debug_invariants_hold(orc, dtype):
    rng = np.random.default_rng(15)
    n, D, R = 400, 16, 8
    x = (rng.integers(0, 256, (n, D), dtype=np.uint8) if dtype == "u8"
         else rng.standard_normal((n, D)).astype(np.float32))
    g = random_graph(rng, n, R, sentinel_frac=0.15)
    ix = orc.pack(x, g)
    qs = x[rng.choice(n, 30)] if dtype == "u8" else rng.standard_normal((30, D)).astype(np.float32)
    for k, L, W in ((1, 1, 1), (10, 10, 3), (10, 33, 4), (16, 64, 16), (8, 20, 64)):
        ix.search(qs, k, L, W, orc.medoid(x), debug=True)   # raises on a violated invariant


def test_adjacency_order_invariance(orc):
    rng = np.random.default_rng(16)
    n, D, R = 500, 16, 10
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    g = random_graph(rng, n, R)
    gp = np.array([rng.permutation(row) for row in g], np.uint32)
    qs = rng.integers(0, 256, (40, D), dtype=np.uint8)
    e = orc.medoid(x)
    a = orc.pack(x, g).search(qs, 10, 24, 4, e)
    b = orc.pack(x, gp).search(qs, 10, 24, 4, e)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert np.array_equal(a[2], b[2])


def test_layout_invariance(orc):
    rng = np.random.default_rng(17)
    n, D, R = 500, 32, 8
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    g = random_graph(rng, n, R)
    qs = rng.integers(0, 256, (40, D), dtype=np.uint8)
    e = orc.medoid(x)
    ref = orc.pack(x, g).search(qs, 10, 32, 4, e)
    rb = orc.record_bytes(0, D, R)
    for kw in (dict(node_to_slot=rng.permutation(n).astype(np.uint32)),
               dict(record_bytes=rb + 12),
               dict(records_per_page=3),
               dict(page_bytes=8192),
               dict(vectors_first=True),
               dict(vectors_first=True, records_per_page=5, node_to_slot=rng.permutation(n).astype(np.uint32))):
        got = orc.pack(x, g, **kw).search(qs, 10, 32, 4, e)
        for a, b in zip(ref[:3], got[:3]):
            assert np.array_equal(a, b)


def test_L_equal_n_evaluates_whole_component(orc):
    rng = np.random.default_rng(18)
    n, D, R = 300, 8, 5
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    g = random_graph(rng, n, R)
    ix = orc.pack(x, g)
    q = rng.integers(0, 256, (3, D), dtype=np.uint8)
    for W in (1, 3):
        _, _, c, _ = ix.search(q, 1, n, W, 0)
        assert (c["evaluations"] == n).all() and (c["expansions"] == n).all()
