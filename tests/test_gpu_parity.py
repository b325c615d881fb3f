"""GPU parity: the HIP library against the CPU oracle, element by element.

uint8 data: ids and int32 distances must match bit-exact (ties broken by id),
and the per-search counters (expansions, iterations, first-time evaluations)
must equal the oracle's summed counts.

float32 data: both sides sum (q_d - x_d)^2 sequentially in d with every
operation rounded (no fused multiply-add), so distances match bit for bit as
well (compared as uint32 patterns) and so do the ids; the 1e-5 relative
tolerance and 0.999 id overlap are checked first as the acceptance bound,
then exactness.
"""
import ctypes
import json
import os
from pathlib import Path

import numpy as np
import pytest

import paper_2607_04415_amd as g
from conftest import NO_EDGE, random_graph
from workload import IndexSpec, QuerySpec, WORKLOADS, index_arrays, query_array

pytestmark = pytest.mark.gpu

GOLDEN = Path(__file__).parent / "golden"


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    torch.cuda.set_device(0)
    return torch


def run_gpu(torch, ix, q, k, L, W):
    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    ids, dists, st = ix.search(qd, k, L, W)
    torch.cuda.synchronize()
    return ids.cpu().numpy().view(np.uint32), dists.cpu().numpy(), st


def f32_acceptance(gi, gd, oids, od, rel=1e-5, overlap=0.999):
    """The float32 bound: distances within `rel` relative, ids overlapping at
    least `overlap` (per-row set intersection over all rows)."""
    fin = np.isfinite(od)
    assert np.array_equal(np.isfinite(gd), fin)
    assert np.all(np.abs(gd[fin] - od[fin]) <= rel * np.abs(od[fin]))
    common = sum(len(np.intersect1d(a[a != NO_EDGE], b[b != NO_EDGE])) for a, b in zip(gi, oids))
    total = int((oids != NO_EDGE).sum())
    assert total == 0 or common / total >= overlap


def check_parity(orc, torch, x, graph, q, k, L, W, layout=None, entry=None, counts=True):
    layout = layout or {}
    ix = g.Index(x, graph, entry=entry, **layout)
    e = ix.info["entry"]
    if entry is None:
        assert e == orc.medoid(x)
    okw = {kk: v for kk, v in layout.items() if v is not None and not (np.isscalar(v) and v == 0)}
    oids, od, oc, _ = orc.pack(x, graph, **okw).search(q, k, L, W, e, threads=8)
    gi, gd, st = run_gpu(torch, ix, q, k, L, W)
    if gd.dtype == np.float32:
        f32_acceptance(gi, gd, oids, od)
        gd, od = gd.view(np.uint32), od.view(np.uint32)
    bad = np.flatnonzero((gi != oids).any(1) | (gd != od).any(1))
    assert bad.size == 0, f"{bad.size} queries differ, first {bad[:5]}: gpu {gi[bad[0]]} {gd[bad[0]]} " \
                          f"oracle {oids[bad[0]]} {od[bad[0]]}"
    if counts:
        assert st["expansions"] == int(oc["expansions"].sum())
        assert st["iterations"] == int(oc["iterations"].sum())
        assert st["evaluations"] - st["reevaluations"] <= int(oc["evaluations"].sum()) <= st["evaluations"]
        if st["reevaluations"] == 0:
            assert st["evaluations"] == int(oc["evaluations"].sum())
    return ix, st


# --------------------------------------------------------------------------- #
def test_trace8_on_gpu(orc, torch_dev):
    t = json.loads((GOLDEN / "trace8.json").read_text())
    x = np.array(t["vectors"], np.uint8)
    graph = np.array(t["graph"], np.uint32)
    ix = g.Index(x, graph)
    assert ix.info["entry"] == t["medoid"]["entry"]
    for c in t["cases"]:
        gi, gd, st = run_gpu(torch_dev, ix, np.array([c["query"]], np.uint8), c["k"], c["L"], c["W"])
        assert gi[0].tolist() == c["ids"]
        assert gd[0].tolist() == c["dists"]
        assert st["evaluations"] == c["evaluations"]
        assert st["expansions"] == c["expansions"]
        assert st["iterations"] == c["iterations"]


CASES = [
    # n, D, R, clusters, k, L, W
    (1000, 128, 32, 4, 10, 32, 4),
    (777, 64, 20, 3, 5, 50, 3),
    (5000, 128, 64, 8, 10, 64, 4),
    (3000, 16, 100, 6, 16, 100, 7),
    (4000, 256, 48, 5, 20, 200, 16),
    (2000, 512, 16, 4, 1, 1, 1),
    (1500, 32, 24, 3, 12, 256, 256),
    (2500, 4, 8, 2, 8, 65, 2),
]


@pytest.mark.parametrize("case", CASES, ids=[f"n{c[0]}-D{c[1]}-R{c[2]}-k{c[4]}-L{c[5]}-W{c[6]}" for c in CASES])
def test_parity_mixture(orc, torch_dev, case):
    n, D, R, C, k, L, W = case
    spec = IndexSpec(n=n, D=D, dtype="u8", clusters=C, sigma=20.0, r_near=R // 2, r_rand=R - R // 2,
                     seed=100 + n)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(300, 7 + n))
    check_parity(orc, torch_dev, a["x"], a["graph"], q, k, L, W)


def test_parity_random_graph_with_missing_edges(orc, torch_dev):
    rng = np.random.default_rng(1)
    n, D, R = 1200, 32, 40
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    graph = random_graph(rng, n, R, sentinel_frac=0.35)
    q = rng.integers(0, 256, (200, D), dtype=np.uint8)
    check_parity(orc, torch_dev, x, graph, q, 10, 40, 5)


@pytest.mark.parametrize("layout", [
    dict(node_to_slot="perm"), dict(record_bytes=400), dict(records_per_page=3),
    dict(page_bytes=8192), dict(page_bytes=16),
    dict(vectors_first=True), dict(vectors_first=True, node_to_slot="perm", record_bytes=420),
], ids=["perm", "rec400", "rpp3", "page8k", "page16-tiny", "vfirst", "vfirst-perm-rec420"])
def test_parity_layouts(orc, torch_dev, layout):
    layout = {"vectors_first": False, **layout}   # the oracle packs contiguous records unless told otherwise
    rng = np.random.default_rng(2)
    n, D, R = 2000, 128, 64
    if layout.get("page_bytes") == 16:
        D, R = 4, 2
        layout = dict(page_bytes=16, vectors_first=False)
    spec = IndexSpec(n=n, D=D, dtype="u8", clusters=4, sigma=20.0, r_near=R // 2, r_rand=R // 2, seed=5)
    a = index_arrays(spec, use_cache=False)
    if layout.get("node_to_slot") == "perm":
        layout = dict(layout, node_to_slot=rng.permutation(n).astype(np.uint32))
    q = query_array(spec, QuerySpec(150, 3))
    ix, _ = check_parity(orc, torch_dev, a["x"], a["graph"], q, 10, 48, 4, layout=layout)
    okw = {kk: v for kk, v in layout.items() if v is not None and not (np.isscalar(v) and v == 0)}
    want = orc.pack(a["x"], a["graph"], **okw).pages
    assert np.array_equal(ix.pages(), want), "packed pages differ from the oracle's packer"


def test_ties_and_duplicates(orc, torch_dev):
    rng = np.random.default_rng(3)
    base = rng.integers(0, 256, (50, 16), dtype=np.uint8)
    x = base[rng.integers(0, 50, 1000)]           # many identical vectors
    graph = random_graph(rng, 1000, 24)
    q = base[rng.integers(0, 50, 100)]            # queries equal to data points: distance 0 ties
    check_parity(orc, torch_dev, x, graph, q, 16, 64, 4)


def test_unreachable_and_padding(orc, torch_dev):
    x = (np.arange(200, dtype=np.uint32) % 256).astype(np.uint8).reshape(200, 1).repeat(4, 1)
    graph = np.full((200, 3), NO_EDGE, np.uint32)
    for i in range(5):                       # component {0..4}; the rest is unreachable
        graph[i] = [(i + 1) % 5, NO_EDGE, (i + 2) % 5]
    for i in range(5, 200):
        graph[i] = [5 + (i - 4) % 195, NO_EDGE, NO_EDGE]
    q = np.array([[100, 100, 100, 100], [0, 0, 0, 0]], np.uint8)
    ix, _ = check_parity(orc, torch_dev, x, graph, q, 8, 16, 2, entry=0)
    gi, gd, _ = run_gpu(torch_dev, ix, q, 8, 16, 2)
    assert (gi[:, 5:] == NO_EDGE).all() and (gd[:, 5:] == 2 ** 31 - 1).all()


def test_visited_filter_overflow_still_exact(orc, torch_dev):
    """A search that outgrows the visited table forgets nodes: re-evaluations
    happen, results and expansion counts do not change."""
    spec = IndexSpec(n=60000, D=64, dtype="u8", clusters=8, sigma=20.0, r_near=32, r_rand=32, seed=9)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(64, 10))
    _, st = check_parity(orc, torch_dev, a["x"], a["graph"], q, 10, 256, 8)
    assert st["reevaluations"] > 0, "the test did not exercise the overflow path"


def _home_bucket_u8(ids, log2=12):
    """Home bucket of each id in the resident uint8 kernel's 16-bit visited
    table with 2^log2 half-words: the top log2 - 3 bits of
    h = (id * 0x3779B1) mod 2^(log2 + 11) (the hash's 24-bit multiplier)."""
    h = (ids.astype(np.uint64) * 0x3779B1) % (1 << (log2 + 11))
    return (h >> 14).astype(np.int64)


@pytest.mark.parametrize("vectors_first", [False, True])
def test_visited_filter_bucket_collisions(orc, torch_dev, vectors_first):
    """Adjacency lists built to collide in the visited table: 64 neighbours
    that share one home bucket (seven slots fill, the rest take the next
    bucket or go unrecorded), lists of a few ids repeated many times (lanes
    holding the same id), and beams whose lists overlap."""
    rng = np.random.default_rng(77)
    n, D, R = 50000, 128, 64
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    graph = rng.integers(0, n, (n, R), dtype=np.uint32)
    graph[:, 0] = (np.arange(n, dtype=np.uint32) + 1) % n
    home = _home_bucket_u8(np.arange(n))
    buckets = np.bincount(home, minlength=512)
    b = int(np.argmax(buckets))
    same = np.flatnonzero(home == b)
    nxt = np.flatnonzero(home == (b + 1) % 512)
    assert len(same) >= 64 and len(nxt) >= 64
    graph[0] = rng.permutation(same)[:64]                       # one bucket, 64 ids
    for j, v in enumerate(graph[0][:8]):                        # their lists: more of it
        graph[v] = np.concatenate([rng.permutation(same)[:32], rng.permutation(nxt)[:32]])
    for v in graph[0][8:16]:                                    # few ids, many copies
        graph[v] = np.repeat(rng.permutation(same)[:8], 8)
    for v in graph[0][16:24]:                                   # overlapping lists
        graph[v] = graph[graph[0][0]]
    q = rng.integers(0, 256, (96, D), dtype=np.uint8)
    _, st = check_parity(orc, torch_dev, x, graph, q, 10, 64, 4, entry=0,
                         layout=dict(vectors_first=vectors_first))


def test_more_than_2_24_nodes_uses_the_32bit_table(orc, torch_dev):
    """Above 2^24 nodes the resident kernel's 16-bit visited table cannot hold
    every id; the 32-bit table takes over and results stay exact."""
    rng = np.random.default_rng(31)
    n, D, R = (1 << 24) + 4099, 4, 4
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    graph = rng.integers(0, n, (n, R), dtype=np.uint32)
    graph[:, 0] = (np.arange(n, dtype=np.uint64) * 2654435761 % n).astype(np.uint32)  # long jumps
    q = rng.integers(0, 256, (64, D), dtype=np.uint8)
    check_parity(orc, torch_dev, x, graph, q, 10, 64, 4, entry=n - 1)


def test_single_node_and_widest_rows(orc, torch_dev):
    # one node, no edges: the answer is that node, then padding
    x1 = np.array([[7, 8, 9, 10]], np.uint8)
    g1 = np.full((1, 3), NO_EDGE, np.uint32)
    ix = g.Index(x1, g1)
    gi, gd, st = run_gpu(torch_dev, ix, np.array([[7, 8, 9, 11]], np.uint8), 4, 8, 2)
    assert gi[0].tolist() == [0, NO_EDGE, NO_EDGE, NO_EDGE]
    assert gd[0].tolist() == [1, 2 ** 31 - 1, 2 ** 31 - 1, 2 ** 31 - 1]
    assert st["expansions"] == 1 and st["evaluations"] == 1
    # R = 256, the widest adjacency list
    rng = np.random.default_rng(33)
    n, D, R = 700, 16, 256
    x = rng.integers(0, 256, (n, D), dtype=np.uint8)
    graph = random_graph(rng, n, R, sentinel_frac=0.2)
    q = rng.integers(0, 256, (100, D), dtype=np.uint8)
    check_parity(orc, torch_dev, x, graph, q, 10, 64, 4)


def test_host_pointers(orc, torch_dev):
    """Host buffers go through the index's staging buffer: all on the host,
    mixed with device buffers, and batches that shrink and then grow it."""
    torch = torch_dev
    spec = IndexSpec(n=1000, D=32, dtype="u8", clusters=3, sigma=20.0, r_near=8, r_rand=8, seed=11)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(600, 12))
    ix = g.Index(a["x"], a["graph"])
    oids, od, _, _ = orc.pack(a["x"], a["graph"]).search(q, 10, 20, 2, ix.info["entry"])
    ids, dists, st = ix.search(q[:40], 10, 20, 2)     # numpy in -> numpy out
    assert np.array_equal(ids, oids[:40]) and np.array_equal(dists, od[:40])
    for nq, where in ((40, "qdev"), (40, "outdev"), (7, "host"), (600, "host"), (600, "qdev"),
                      (250, "outdev"), (600, "idsdev")):
        qh = np.ascontiguousarray(q[:nq])
        qs = torch.from_numpy(qh).cuda() if where == "qdev" else qh
        ih = np.full((nq, 10), 7, np.uint32)
        dh = np.full((nq, 10), 7, np.int32)
        idd = torch.full((nq, 10), 7, dtype=torch.int32, device="cuda")
        ddd = torch.full((nq, 10), 7, dtype=torch.int32, device="cuda")
        ids_buf = idd if where in ("outdev", "idsdev") else ih
        d_buf = ddd if where == "outdev" else dh
        ix.search_into(qs, nq, 10, 20, 2, ids_buf, d_buf)
        torch.cuda.synchronize()
        got_i = ids_buf.cpu().numpy().view(np.uint32) if ids_buf is idd else ids_buf
        got_d = d_buf.cpu().numpy() if d_buf is ddd else d_buf
        assert np.array_equal(got_i, oids[:nq]), (nq, where)
        assert np.array_equal(got_d, od[:nq]), (nq, where)
    ix.close()


def test_empty_batch_and_bad_arguments(torch_dev):
    spec = IndexSpec(n=500, D=16, dtype="u8", clusters=2, sigma=20.0, r_near=4, r_rand=4, seed=13)
    a = index_arrays(spec, use_cache=False)
    ix = g.Index(a["x"], a["graph"])
    q = np.zeros((1, 16), np.uint8)
    assert ix.search_into(q, 0, 1, 1, 1, None, None) is not None          # nq = 0: no-op
    for k, L, W in ((0, 4, 1), (5, 4, 1), (1, 257, 1), (1, 4, 0), (1, 4, 5)):
        with pytest.raises(g.GorioError) as e:
            ix.search(q, k, L, W)
        assert e.value.status == g.EINVAL
    # buffers the search would overrun are refused before the library sees them
    torch = torch_dev
    qd = torch.zeros((4, 16), dtype=torch.uint8, device="cuda")
    small = torch.empty((3, 1), dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError):
        ix.search_into(qd, 4, 1, 4, 1, small, small)
    with pytest.raises(ValueError):
        ix.search_into(qd[:3], 4, 1, 4, 1, small, small)
    with pytest.raises(ValueError):
        ix.search(np.zeros((2, 15), np.uint8), 1, 4, 1)
    ids, dists, _ = ix.search(qd, 1, 4, 1)        # the index is still usable
    assert ids.shape == (4, 1)


F32_CASES = [
    # n, D, R, clusters, k, L, W
    (2000, 96, 32, 4, 10, 64, 4),
    (3000, 96, 64, 8, 10, 128, 8),        # the 10M workload's shape at a small n
    (1500, 37, 24, 3, 12, 100, 5),        # generic path, D not a multiple of 4
    (1000, 256, 16, 4, 5, 200, 16),
    (800, 1, 8, 2, 4, 16, 2),
    (1200, 20, 40, 3, 256, 256, 64),
]


@pytest.mark.parametrize("case", F32_CASES,
                         ids=[f"n{c[0]}-D{c[1]}-R{c[2]}-k{c[4]}-L{c[5]}-W{c[6]}" for c in F32_CASES])
def test_parity_f32_mixture(orc, torch_dev, case):
    n, D, R, C, k, L, W = case
    spec = IndexSpec(n=n, D=D, dtype="f32", clusters=C, sigma=0.05, r_near=R // 2, r_rand=R - R // 2,
                     seed=300 + n)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(300, 17 + n))
    check_parity(orc, torch_dev, a["x"], a["graph"], q, k, L, W)


def test_parity_f32_layout_perm_and_wide_records(orc, torch_dev):
    rng = np.random.default_rng(21)
    spec = IndexSpec(n=2500, D=96, dtype="f32", clusters=5, sigma=0.05, r_near=32, r_rand=32, seed=22)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(200, 23))
    for layout in (dict(node_to_slot=rng.permutation(2500).astype(np.uint32)), dict(record_bytes=700),
                   dict(page_bytes=8192, records_per_page=5), dict(vectors_first=True)):
        check_parity(orc, torch_dev, a["x"], a["graph"], q, 10, 128, 8, layout=layout)


def test_f32_ties_zero_distance_and_padding(orc, torch_dev):
    rng = np.random.default_rng(24)
    base = rng.standard_normal((40, 12)).astype(np.float32)
    x = base[rng.integers(0, 40, 900)]                # identical vectors: equal distances
    graph = random_graph(rng, 900, 16, sentinel_frac=0.2)
    q = np.concatenate([base[:20], rng.standard_normal((20, 12)).astype(np.float32)])
    check_parity(orc, torch_dev, x, graph, q, 16, 64, 4)
    # a 5-node component: the tail of every row is padding (+inf)
    x2 = rng.standard_normal((50, 8)).astype(np.float32)
    g2 = np.full((50, 2), NO_EDGE, np.uint32)
    for i in range(5):
        g2[i] = [(i + 1) % 5, (i + 3) % 5]
    ix, _ = check_parity(orc, torch_dev, x2, g2, x2[:3], 8, 16, 2, entry=0)
    gi, gd, _ = run_gpu(torch_dev, ix, x2[:3], 8, 16, 2)
    assert (gi[:, 5:] == NO_EDGE).all() and np.isposinf(gd[:, 5:]).all()


def test_f32_visited_filter_overflow_still_exact(orc, torch_dev):
    spec = IndexSpec(n=60000, D=16, dtype="f32", clusters=8, sigma=0.05, r_near=32, r_rand=32, seed=25)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(48, 26))
    _, st = check_parity(orc, torch_dev, a["x"], a["graph"], q, 10, 256, 8)
    assert st["reevaluations"] > 0, "the test did not exercise the overflow path"


def test_entry_rule_matches_oracle_f32(orc, torch_dev):
    rng = np.random.default_rng(14)
    x = rng.standard_normal((3000, 96)).astype(np.float32)
    graph = random_graph(rng, 3000, 8)
    ix = g.Index(x, graph, vectors_first=False)
    assert ix.info["entry"] == orc.medoid(x)
    assert np.array_equal(ix.pages(), orc.pack(x, graph).pages)


# --------------------------------------------------------------------------- #
# benchmark workloads at full size
# --------------------------------------------------------------------------- #
def _workload_parity(orc, torch, name, threads=16):
    w = WORKLOADS[name]
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)
    print(f"[{name}] n={w.index.n} nq={len(q)} k={w.k} L={w.L} W={w.W}", flush=True)
    ix = g.Index(a["x"], a["graph"])     # the library's default arrangement: vectors first
    assert ix.info["vectors_first"] == 1
    e = ix.info["entry"]
    assert e == orc.medoid(a["x"])
    packed = orc.pack(a["x"], a["graph"], vectors_first=True)
    assert np.array_equal(ix.pages(), packed.pages)
    oids, od, oc, _ = packed.search(q, w.k, w.L, w.W, e, threads=threads)
    gi, gd, st = run_gpu(torch, ix, q, w.k, w.L, w.W)
    assert np.array_equal(gi, oids) and np.array_equal(gd, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    assert st["evaluations"] - st["reevaluations"] <= int(oc["evaluations"].sum())
    print(f"[{name}] bit-exact; kernel {st['kernel_ms']:.3f} ms; evals {st['evaluations']} "
          f"(re {st['reevaluations']}) oracle {int(oc['evaluations'].sum())}", flush=True)


def test_workload_u8_10k(orc, torch_dev):
    _workload_parity(orc, torch_dev, "u8-10k-hbm")


def test_workload_u8_1m(orc, torch_dev):
    _workload_parity(orc, torch_dev, "u8-1m-hbm")


@pytest.mark.parametrize("seed", range(12))
def test_resident_random_configuration(orc, torch_dev, seed):
    """Seeded random resident configurations: dtype, sizes, beam, page layout."""
    rng = np.random.default_rng(2000 + seed)
    dtype = "u8" if rng.random() < 0.6 else "f32"
    D = int(rng.choice([4, 8, 32, 128, 256]) if dtype == "u8" else rng.choice([3, 24, 96, 160]))
    R = int(rng.choice([4, 16, 40, 64, 128]))
    n = int(rng.integers(max(R + 2, 500), 20000))
    spec = IndexSpec(n=n, D=D, dtype=dtype, clusters=int(rng.integers(1, 9)),
                     sigma=20.0 if dtype == "u8" else 0.05, r_near=R // 2, r_rand=R - R // 2,
                     seed=int(rng.integers(1 << 30)))
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(int(rng.integers(20, 400)), int(rng.integers(1 << 30))))
    L = int(rng.choice([1, 8, 33, 64, 65, 128, 200, 256]))
    k = int(rng.integers(1, L + 1))
    W = int(rng.integers(1, L + 1)) if rng.random() < 0.2 else int(rng.integers(1, min(L, 16) + 1))
    layout = dict(vectors_first=bool(rng.random() < 0.5))
    if rng.random() < 0.3:
        layout["node_to_slot"] = rng.permutation(n).astype(np.uint32)
    if rng.random() < 0.2:
        layout["page_bytes"] = 8192
    print(f"[resident random {seed}] {dtype} n={n} D={D} R={R} k={k} L={L} W={W} "
          f"vfirst={layout['vectors_first']} perm={'node_to_slot' in layout} page={layout.get('page_bytes', 4096)}",
          flush=True)
    check_parity(orc, torch_dev, a["x"], a["graph"], q, k, L, W,
                 layout={kk: v for kk, v in layout.items()})


def test_searches_on_two_streams_do_not_share_counters(orc, torch_dev):
    """Two searches of one index queued back to back on different streams
    without waiting (device buffers, no stats): each must write every row.
    They share the index's query counter, so the library orders the second
    after the first on the GPU."""
    torch = torch_dev
    spec = IndexSpec(n=30000, D=128, dtype="u8", clusters=8, sigma=20.0, r_near=16, r_rand=16, seed=91)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(6000, 92))
    k, L, W = 10, 48, 4
    ix = g.Index(a["x"], a["graph"])
    ref_ids, ref_d, _ = run_gpu(torch, ix, q, k, L, W)
    qd = torch.from_numpy(q).cuda()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = [(torch.full((len(q), k), -1, dtype=torch.int32, device="cuda"),
             torch.full((len(q), k), -1, dtype=torch.int32, device="cuda")) for _ in range(4)]
    torch.cuda.synchronize()          # the buffers are filled before either stream writes them
    for s, (ids, dd) in zip((s1, s2, s1, s2), outs):
        ix.search_into(qd, len(q), k, L, W, ids, dd, stream=s.cuda_stream, stats=False)
    torch.cuda.synchronize()
    for ids, dd in outs:
        assert np.array_equal(ids.cpu().numpy().view(np.uint32), ref_ids)
        assert np.array_equal(dd.cpu().numpy(), ref_d)
    ix.close()


def test_stream_created_after_another_is_destroyed(orc, torch_dev):
    """A stream created after another was destroyed may get its handle; on
    created streams the index always waits for its last search's event (here
    one recorded on a stream since destroyed), and each search answers every
    query.  Each stream is synchronized before it is destroyed."""
    torch = torch_dev
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    spec = IndexSpec(n=20000, D=128, dtype="u8", clusters=8, sigma=20.0, r_near=16, r_rand=16, seed=97)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(2000, 98))
    k, L, W = 10, 32, 4
    ix = g.Index(a["x"], a["graph"])
    ref_ids, ref_d, _ = run_gpu(torch, ix, q, k, L, W)
    qd = torch.from_numpy(q).cuda()
    ids = torch.full((len(q), k), -1, dtype=torch.int32, device="cuda")
    dd = torch.full((len(q), k), -1, dtype=torch.int32, device="cuda")
    for _ in range(3):
        s = ctypes.c_void_p()
        assert hip.hipStreamCreate(ctypes.byref(s)) == 0
        ids.fill_(-1)
        dd.fill_(-1)
        torch.cuda.synchronize()
        ix.search_into(qd, len(q), k, L, W, ids, dd, stream=s.value, stats=False)
        assert hip.hipStreamSynchronize(s) == 0
        assert hip.hipStreamDestroy(s) == 0
        assert np.array_equal(ids.cpu().numpy().view(np.uint32), ref_ids)
        assert np.array_equal(dd.cpu().numpy(), ref_d)
    ix.close()


def test_back_to_back_searches_without_stats_then_with(orc, torch_dev):
    """The query-ticket counter and the statistics counters are never reset
    between searches: searches of different sizes queued back to back without
    statistics (one stream, then a second), and a paged search in between, must
    each answer every query exactly; a search that asks for statistics then
    reports its own counts only (the oracle's expansions and iterations)."""
    torch = torch_dev
    spec = IndexSpec(n=20000, D=128, dtype="u8", clusters=8, sigma=20.0, r_near=16, r_rand=16, seed=95)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(3000, 96))
    k, L, W = 10, 32, 4
    ix = g.Index(a["x"], a["graph"])
    e = ix.info["entry"]
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, k, L, W, e, threads=16)
    qd = torch.from_numpy(q).cuda()
    sizes = [3000, 1, 1777, 3000, 64, 2500]
    outs = [(torch.full((m, k), -1, dtype=torch.int32, device="cuda"),
             torch.full((m, k), -1, dtype=torch.int32, device="cuda")) for m in sizes]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for i, (m, (ids, dd)) in enumerate(zip(sizes, outs)):
        s = s1 if i < 4 else s2
        ix.search_into(qd[:m], m, k, L, W, ids, dd, stream=s.cuda_stream, stats=False)
    torch.cuda.synchronize()
    for m, (ids, dd) in zip(sizes, outs):
        assert np.array_equal(ids.cpu().numpy().view(np.uint32), oids[:m]), m
        assert np.array_equal(dd.cpu().numpy(), od[:m]), m
    gi, gd, st = run_gpu(torch, ix, q, k, L, W)
    assert np.array_equal(gi, oids) and np.array_equal(gd, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    assert st["iterations"] == int(oc["iterations"].sum())
    # a paged search on the same index, then resident again: counts stay per search
    ix.set_cache(int(0.2 * ix.info["index_bytes"]))
    pi, pd, pst = run_gpu(torch, ix, q[:500], k, L, W)
    assert np.array_equal(pi, oids[:500]) and np.array_equal(pd, od[:500])
    assert pst["expansions"] == int(oc["expansions"][:500].sum())
    ix.set_cache(ix.info["index_bytes"])
    gi, gd, st = run_gpu(torch, ix, q[:2000], k, L, W)
    assert np.array_equal(gi, oids[:2000]) and np.array_equal(gd, od[:2000])
    assert st["expansions"] == int(oc["expansions"][:2000].sum())
    ix.close()


@pytest.mark.timeout(900)
@pytest.mark.skipif(os.environ.get("GORIO_SKIP_BIG") == "1", reason="GORIO_SKIP_BIG=1: a 4.3 GB index")
def test_index_above_4gib_is_exact(orc, torch_dev):
    """A uint8 128-d index whose pages span more than 4 GiB (one 4 KB record
    per page): vectors can no longer be named by 32-bit buffer offsets, so the
    kernel must address them with 64-bit pointers; answers equal the oracle's."""
    spec = IndexSpec(n=1_050_000, D=128, dtype="u8", clusters=16, sigma=20.0, r_near=8, r_rand=8, seed=93)
    a = index_arrays(spec)
    q = query_array(spec, QuerySpec(300, 94))
    layout = dict(vectors_first=True, record_bytes=4096)
    ix = g.Index(a["x"], a["graph"], **layout)
    assert ix.info["index_bytes"] > (1 << 32)
    e = ix.info["entry"]
    gi, gd, st = run_gpu(torch_dev, ix, q, 10, 32, 4)
    ix.close()
    oids, od, oc, _ = orc.pack(a["x"], a["graph"], **layout).search(q, 10, 32, 4, e, threads=16)
    assert np.array_equal(gi, oids) and np.array_equal(gd, od)
    assert st["expansions"] == int(oc["expansions"].sum())
