"""GPU parity of the paged search (HBM page cache + host backing store + proxy).

Results must equal the CPU oracle bit-exact whatever the cache size, the
injected latency, the query-slot oversubscription or the blocking mode
(float32 distances compared as uint32 bit patterns).
"""
import numpy as np
import pytest

import paper_2607_04415_amd as g

from workload import IndexSpec, QuerySpec, WORKLOADS, index_arrays, query_array

pytestmark = pytest.mark.gpu

SPEC = IndexSpec(n=20000, D=128, dtype="u8", clusters=8, sigma=20.0, r_near=16, r_rand=16, seed=41)


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    torch.cuda.set_device(0)
    return torch


@pytest.fixture(scope="module")
def small(orc):
    a = index_arrays(SPEC, use_cache=False)
    q = query_array(SPEC, QuerySpec(400, 42))
    e = orc.medoid(a["x"])
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, 10, 32, 4, e, threads=8)
    return a, q, oids, od, oc


def search(torch, ix, q, k, L, W):
    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    ids, dists, st = ix.search(qd, k, L, W)
    torch.cuda.synchronize()
    return ids.cpu().numpy().view(np.uint32), dists.cpu().numpy(), st


def assert_same(gi, gd, oids, od):
    if gd.dtype == np.float32:
        gd, od = gd.view(np.uint32), od.view(np.uint32)
    bad = np.flatnonzero((gi != oids).any(1) | (gd != od).any(1))
    assert bad.size == 0, f"{bad.size} queries differ, first {bad[:5]}"


@pytest.mark.parametrize("frac,latency,oversub,blocking,vfirst", [
    (0.10, 0.0, 1, 0, 0), (0.10, 20.0, 4, 0, 0), (0.30, 0.0, 2, 0, 0), (0.10, 0.0, 1, 1, 0),
    (0.50, 5.0, 8, 0, 0), (0.10, 20.0, 4, 0, 1),
], ids=["c10-l0-o1", "c10-l20-o4", "c30-l0-o2", "c10-l0-blocking", "c50-l5-o8", "c10-l20-o4-vfirst"])
def test_paged_matches_oracle(torch_dev, small, frac, latency, oversub, blocking, vfirst):
    a, q, oids, od, oc = small
    ix = g.Index(a["x"], a["graph"], vectors_first=bool(vfirst))
    info = ix.info
    ix.set_cache(max(int(frac * info["index_bytes"]), 128 * 4096))
    ix.set_backing(latency_us=latency, oversub=oversub, blocking=bool(blocking))
    assert not ix.info["resident"]
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    assert st["iterations"] == int(oc["iterations"].sum())
    assert st["misses"] > 0 and st["pages_served"] > 0
    # every record access was either a hit or a miss
    assert st["hits"] + st["misses"] == st["expansions"] + st["evaluations"]
    assert st["bytes_served"] == st["pages_served"] * 4096
    assert st["parks"] > 0


def test_paged_tiny_cache_slot_reuse(torch_dev, small):
    """The smallest cache (128 slots): every slot is reused many times."""
    a, q, oids, od, _ = small
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(128 * 4096)
    ix.set_backing(latency_us=0.0, oversub=1)
    assert ix.info["cache_slots"] == 128
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["pages_served"] > 10 * 128


def test_warm_cache_second_search(orc, torch_dev):
    """A cache that never has to evict: the second search over the same
    queries finds every page resident (no misses) and returns the same answers."""
    spec = IndexSpec(n=200000, D=128, dtype="u8", clusters=16, sigma=20.0, r_near=16, r_rand=16, seed=43)
    a = index_arrays(spec)
    q = query_array(spec, QuerySpec(4, 44))
    e = orc.medoid(a["x"])
    oids, od, _, _ = orc.pack(a["x"], a["graph"]).search(q, 10, 32, 4, e)
    ix = g.Index(a["x"], a["graph"])
    nearly_all = int(0.95 * ix.info["index_bytes"])    # far more slots than 4 queries touch
    ix.set_cache(nearly_all)
    s1 = search(torch_dev, ix, q, 10, 32, 4)
    s2 = search(torch_dev, ix, q, 10, 32, 4)           # cache carries over
    for gi, gd, _ in (s1, s2):
        assert_same(gi, gd, oids, od)
    assert s1[2]["misses"] > 0
    assert s2[2]["misses"] == 0 and s2[2]["pages_served"] == 0
    assert s2[2]["hits"] == s1[2]["hits"] + s1[2]["misses"]
    ix.set_cache(nearly_all)                            # empties it again
    s3 = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(s3[0], s3[1], oids, od)
    # cold again (exact counts vary: a page two queries want at once is a
    # miss for both or a hit for the later one, depending on timing)
    assert s3[2]["misses"] > s1[2]["misses"] // 2


def test_paged_to_resident_and_back(torch_dev, small):
    a, q, oids, od, _ = small
    ix = g.Index(a["x"], a["graph"])
    pages = ix.pages()
    ix.set_cache(200 * 4096)
    assert np.array_equal(ix.pages(), pages)            # backing store holds the same bytes
    ix.set_cache(ix.info["index_bytes"])
    assert ix.info["resident"]
    gi, gd, _ = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)


def test_paged_rejects(torch_dev, small):
    a, q, _, _, _ = small
    ix = g.Index(a["x"], a["graph"])
    with pytest.raises(g.GorioError) as e:
        ix.set_cache(10 * 4096)                          # fewer than two queries' worth of pins
    assert e.value.status == g.EINVAL
    ix.set_cache(300 * 4096)
    with pytest.raises(g.GorioError) as e:
        ix.search(q[:4], 10, 128, 65)                    # paged search takes W <= 64
    assert e.value.status == g.EUNSUPPORTED
    with pytest.raises(g.GorioError):
        ix.set_backing(oversub=0)


def test_watchdog_abort_then_recover(torch_dev, small, monkeypatch):
    """The host trips the watchdog at once: the kernel exits, the call reports
    a time-out, and the next search runs normally."""
    a, q, oids, od, _ = small
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(300 * 4096)
    ix.set_backing(latency_us=50.0)
    monkeypatch.setenv("GORIO_WATCHDOG_S", "0")
    with pytest.raises(g.GorioError) as e:
        search(torch_dev, ix, q, 10, 32, 4)
    assert e.value.status == g.ETIMEOUT
    monkeypatch.delenv("GORIO_WATCHDOG_S")
    ix.set_backing(latency_us=0.0)
    gi, gd, _ = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)


@pytest.mark.parametrize("layout", [
    dict(page_bytes=8192), dict(page_bytes=2048), dict(node_to_slot="perm"),
    dict(node_to_slot="perm", vectors_first=True, page_bytes=8192),
], ids=["page8k", "page2k", "perm", "perm-vfirst-page8k"])
def test_paged_layouts(orc, torch_dev, layout):
    """Pages other than 4 KB take the generic copy path; a placement
    permutation takes the node-to-slot branch of every cache address."""
    a = index_arrays(SPEC, use_cache=False)
    q = query_array(SPEC, QuerySpec(200, 49))
    if layout.get("node_to_slot") == "perm":
        layout = dict(layout, node_to_slot=np.random.default_rng(50).permutation(SPEC.n).astype(np.uint32))
    ix = g.Index(a["x"], a["graph"], **layout)
    e = ix.info["entry"]
    oids, od, _, _ = orc.pack(a["x"], a["graph"], **layout).search(q, 10, 32, 4, e, threads=8)
    ix.set_cache(max(int(0.10 * ix.info["index_bytes"]), 128 * ix.info["page_bytes"]))
    ix.set_backing(latency_us=5.0, oversub=4)
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["bytes_served"] == st["pages_served"] * ix.info["page_bytes"]


def test_paged_widest_beam(orc, torch_dev):
    """L = 256 (four frontier slots per lane) and W = 64, the paged kernel's limit."""
    spec = IndexSpec(n=8000, D=32, dtype="u8", clusters=4, sigma=20.0, r_near=24, r_rand=24, seed=51)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(64, 52))
    ix = g.Index(a["x"], a["graph"])
    e = ix.info["entry"]
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, 100, 256, 64, e, threads=8)
    ix.set_cache(max(int(0.2 * ix.info["index_bytes"]), 256 * 4096))
    ix.set_backing(latency_us=2.0, oversub=2)
    gi, gd, st = search(torch_dev, ix, q, 100, 256, 64)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())


def test_reordered_completions_same_answers(torch_dev, small, monkeypatch):
    """The proxy adds a random 0-100 us delay per request, so pages arrive out
    of request order; the answers do not change."""
    a, q, oids, od, oc = small
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(max(int(0.10 * ix.info["index_bytes"]), 128 * 4096))
    ix.set_backing(latency_us=5.0, oversub=4)
    monkeypatch.setenv("GORIO_PROXY_JITTER_US", "100")
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())


def test_held_proxy_trips_watchdog_then_recovers(torch_dev, small, monkeypatch):
    """A proxy that never completes: the kernel ends at the watchdog with
    GORIO_ETIMEOUT instead of hanging, and the next search is normal."""
    a, q, oids, od, _ = small
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(300 * 4096)
    ix.set_backing(latency_us=0.0)
    monkeypatch.setenv("GORIO_PROXY_HOLD", "1")
    monkeypatch.setenv("GORIO_WATCHDOG_S", "1")
    with pytest.raises(g.GorioError) as e:
        search(torch_dev, ix, q, 10, 32, 4)
    assert e.value.status == g.ETIMEOUT
    assert e.value.stats["pages_served"] == 0
    monkeypatch.delenv("GORIO_PROXY_HOLD")
    monkeypatch.delenv("GORIO_WATCHDOG_S")
    gi, gd, _ = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)


def test_paged_1m_index_slice(orc, torch_dev):
    """The 1M-vector index with a 10% cache, on the first 2,000 queries."""
    w = WORKLOADS["u8-1m-cache10-lat0"]
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)[:2000]
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(int(0.10 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=0.0, oversub=1)
    gi, gd, st = search(torch_dev, ix, q, w.k, w.L, w.W)
    e = ix.info["entry"]
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, w.k, w.L, w.W, e, threads=16)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    hr = st["hits"] / max(1, st["hits"] + st["misses"])
    print(f"[1m paged] {st['kernel_ms']:.1f} ms, hit rate {hr:.3f}, served {st['pages_served']}, "
          f"{st['bytes_served'] / st['kernel_ms'] / 1e6:.2f} GB/s", flush=True)


@pytest.mark.parametrize("name,oversub,waves", [("u8-1m-cache10-lat0", 1, 30), ("u8-1m-cache10-lat20", 4, 30)])
def test_paged_1m_bench_configuration(orc, torch_dev, name, oversub, waves):
    """The benchmark's paged legs at full size and in its launch configuration
    (vectors-first pages placed by 512 clusters, queries admitted by cluster,
    cold 10% cache, the workload's latency, the bench's scheduler shape):
    every query of the configuration equals the oracle."""
    w = WORKLOADS[name]
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)
    n2s, cent = g.cluster_order(a["x"], 512)
    ix = g.Index(a["x"], a["graph"], vectors_first=True, node_to_slot=n2s)
    ix.set_cache(int(w.cache_frac * ix.info["index_bytes"]))
    ix.set_backing(latency_us=w.latency_us, oversub=oversub)
    ix.set_scheduler(query_waves=waves)
    ix.set_query_order(cent)
    gi, gd, st = search(torch_dev, ix, q, w.k, w.L, w.W)
    e = ix.info["entry"]
    ix.close()
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, w.k, w.L, w.W, e, threads=16)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    hr = st["hits"] / max(1, st["hits"] + st["misses"])
    print(f"[{name}] {len(q)} queries, {st['kernel_ms']:.0f} ms, hit rate {hr:.3f}", flush=True)


F32_SPEC = IndexSpec(n=12000, D=96, dtype="f32", clusters=8, sigma=0.05, r_near=32, r_rand=32, seed=45)


@pytest.fixture(scope="module")
def small_f32(orc):
    a = index_arrays(F32_SPEC, use_cache=False)
    q = query_array(F32_SPEC, QuerySpec(300, 46))
    e = orc.medoid(a["x"])
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, 10, 128, 8, e, threads=8)
    return a, q, oids, od, oc


@pytest.mark.parametrize("frac,latency,oversub,blocking", [
    (0.05, 20.0, 4, 0), (0.10, 0.0, 1, 1), (0.30, 5.0, 8, 0),
], ids=["c5-l20-o4", "c10-l0-blocking", "c30-l5-o8"])
def test_paged_f32_matches_oracle(torch_dev, small_f32, frac, latency, oversub, blocking):
    a, q, oids, od, oc = small_f32
    ix = g.Index(a["x"], a["graph"], vectors_first=blocking == 0 and oversub == 8)
    ix.set_cache(max(int(frac * ix.info["index_bytes"]), 128 * 4096))
    ix.set_backing(latency_us=latency, oversub=oversub, blocking=bool(blocking))
    gi, gd, st = search(torch_dev, ix, q, 10, 128, 8)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    assert st["iterations"] == int(oc["iterations"].sum())
    assert st["hits"] + st["misses"] == st["expansions"] + st["evaluations"]
    assert st["misses"] > 0


def test_paged_f32_generic_dims(orc, torch_dev):
    spec = IndexSpec(n=6000, D=37, dtype="f32", clusters=4, sigma=0.05, r_near=12, r_rand=12, seed=47)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(200, 48))
    e = orc.medoid(a["x"])
    oids, od, _, _ = orc.pack(a["x"], a["graph"]).search(q, 10, 64, 4, e, threads=8)
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(max(int(0.1 * ix.info["index_bytes"]), 128 * 4096))
    ix.set_backing(latency_us=0.0, oversub=4)
    gi, gd, _ = search(torch_dev, ix, q, 10, 64, 4)
    assert_same(gi, gd, oids, od)


RANDOM_CONFIGS = 22
QUEUE_FROM = 16      # seeds from here on run the GPU resume queue


@pytest.mark.parametrize("seed", range(RANDOM_CONFIGS))
def test_paged_random_configuration(orc, torch_dev, monkeypatch, seed):
    """Seeded random configurations of the whole paged path: dtype, sizes,
    beam, page size and layout, cache size, latency, slots, scheduling mode
    (split-phase, blocking, host-scheduled lanes run by the executor or by
    a launch per round, or, from seed QUEUE_FROM on, the GPU resume queue)."""
    rng = np.random.default_rng(1000 + seed)
    dtype = "u8" if rng.random() < 0.6 else "f32"
    D = int(rng.choice([4, 16, 64, 128]) if dtype == "u8" else rng.choice([7, 32, 96]))
    R = int(rng.choice([8, 24, 64]))
    n = int(rng.integers(3000, 15000))
    spec = IndexSpec(n=n, D=D, dtype=dtype, clusters=int(rng.integers(2, 9)),
                     sigma=20.0 if dtype == "u8" else 0.05, r_near=R // 2, r_rand=R - R // 2,
                     seed=int(rng.integers(1 << 30)))
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(int(rng.integers(50, 300)), int(rng.integers(1 << 30))))
    L = int(rng.choice([16, 48, 64, 100, 128]))
    k = int(rng.integers(1, min(L, 20) + 1))
    W = int(rng.integers(1, min(L, 16) + 1))
    layout = dict(page_bytes=int(rng.choice([4096, 4096, 8192])), vectors_first=bool(rng.random() < 0.5))
    if rng.random() < 0.3:
        layout["node_to_slot"] = rng.permutation(n).astype(np.uint32)
    # cluster placement and ordered admission (their own stream of draws, so
    # the other parameters of each seed stay as they were)
    crng = np.random.default_rng(5000 + seed)
    cent = None
    if "node_to_slot" not in layout and crng.random() < 0.4:
        layout["node_to_slot"], cent = g.cluster_order(a["x"], int(crng.integers(1, 40)),
                                                       iterations=int(crng.integers(0, 5)))
    ix = g.Index(a["x"], a["graph"], **layout)
    if cent is not None and crng.random() < 0.75:
        ix.set_query_order(cent)
    e = ix.info["entry"]
    oids, od, oc, _ = orc.pack(a["x"], a["graph"], **layout).search(q, k, L, W, e, threads=8)
    pb = ix.info["page_bytes"]
    ix.set_cache(max(int(rng.uniform(0.02, 0.6) * ix.info["index_bytes"]), 128 * pb))
    blocking = bool(rng.random() < 0.25)
    # host-scheduled lanes (their own stream of draws too)
    hrng = np.random.default_rng(9000 + seed)
    queue = seed >= QUEUE_FROM
    host = bool(hrng.random() < 0.35) and not queue
    mode = 3 if queue else (2 if host else int(blocking))
    host_desc = ""
    if queue:
        qrng = np.random.default_rng(13000 + seed)
        ix.set_scheduler(query_waves=int(qrng.choice([0, 1, 3, 16, 40])))
        host_desc = " gpu resume queue"
    if host:
        executor = bool(hrng.random() < 0.6)
        passes = [None, "1", "3"][int(hrng.integers(0, 3))]
        monkeypatch.setenv("GORIO_HOST_EXECUTOR", "1" if executor else "0")
        if passes is not None:
            monkeypatch.setenv("GORIO_TURN_PASSES", passes)
        ix.set_scheduler(query_waves=int(hrng.choice([0, 1, 3, 16])))
        host_desc = f" host executor={executor} passes={passes}"
    ix.set_backing(latency_us=float(rng.choice([0.0, 3.0, 20.0])), oversub=int(rng.choice([1, 2, 4, 8])),
                   mode=mode)
    print(f"[random {seed}] {dtype} n={n} D={D} R={R} k={k} L={L} W={W} {layout.get('page_bytes')} "
          f"vfirst={layout['vectors_first']} perm={'node_to_slot' in layout} clusters={cent is not None} "
          f"slots={ix.info['cache_slots']} mode={mode}{host_desc}", flush=True)
    gi, gd, st = search(torch_dev, ix, q, k, L, W)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())


# --------------------------------------------------------------------------- #
# cluster placement and cluster-ordered admission
# --------------------------------------------------------------------------- #
def test_cluster_order_places_clusters_contiguously(torch_dev):
    """gorio_cluster_order: a permutation that lists the nodes grouped by their
    nearest returned centroid (checked in float64, near-ties excepted), with
    centroids inside the data's range; deterministic."""
    rng = np.random.default_rng(5)
    K, per, D = 8, 1500, 32
    centres = rng.uniform(30, 225, (K, D))
    lab = np.repeat(np.arange(K), per)
    rng.shuffle(lab)
    x = np.clip(np.rint(centres[lab] + 4 * rng.standard_normal((K * per, D))), 0, 255).astype(np.uint8)
    for clusters in (8, 32):
        n2s, cent = g.cluster_order(x, clusters, iterations=6)
        assert np.array_equal(np.sort(n2s), np.arange(len(x), dtype=np.uint32))
        assert cent.shape == (clusters, D) and np.isfinite(cent).all()
        assert (cent >= 0).all() and (cent <= 255).all()
        d = ((x.astype(np.float64)[:, None, :] - cent.astype(np.float64)[None]) ** 2).sum(2)
        srt = np.sort(d, axis=1)
        clear = srt[:, 1] - srt[:, 0] > 1e-3 * np.maximum(srt[:, 0], 1.0)
        key = np.argmin(d, axis=1)[np.argsort(n2s)]
        ok = clear[np.argsort(n2s)]
        kk = key[ok]
        assert (np.diff(kk) >= 0).all(), "slots are not grouped by nearest centroid"
        n2s2, cent2 = g.cluster_order(x, clusters, iterations=6)
        assert np.array_equal(n2s, n2s2) and np.array_equal(cent, cent2)
    # with more centroids than blobs, each cluster stays inside one blob
    by_slot = lab[np.argsort(n2s)]
    runs = 1 + int((by_slot[1:] != by_slot[:-1]).sum())
    assert runs <= 32, runs


@pytest.mark.parametrize("vfirst,blocking", [(True, False), (False, False), (True, True)])
def test_paged_cluster_placement_and_query_order(orc, torch_dev, small, vfirst, blocking):
    """Cluster placement plus cluster-ordered admission: answers equal the
    oracle's (which packs with the same placement) and the plain search's."""
    a, q, oids, od, oc = small
    n2s, cent = g.cluster_order(a["x"], 16)
    ix = g.Index(a["x"], a["graph"], node_to_slot=n2s, vectors_first=vfirst)
    assert ix.info["entry"] == orc.medoid(a["x"])
    ix.set_cache(int(0.15 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=2.0, oversub=1 if blocking else 4, blocking=blocking)
    ix.set_query_order(cent)
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["misses"] > 0
    ix.set_query_order(None)                       # index order again
    gi, gd, _ = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    ix.close()


def test_query_order_resident_and_empty_batch(orc, torch_dev, small):
    """The order is ignored by resident searches; nq = 0 is a no-op."""
    a, q, oids, od, oc = small
    _, cent = g.cluster_order(a["x"], 4, iterations=1)
    ix = g.Index(a["x"], a["graph"])
    ix.set_query_order(cent)
    gi, gd, _ = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    ix.set_cache(int(0.2 * ix.info["index_bytes"]))
    ix.set_backing(oversub=2)
    gi, gd, _ = search(torch_dev, ix, q[:0], 10, 32, 4)
    assert gi.shape == (0, 10)
    ix.close()


def test_paged_f32_cluster_placement_and_query_order(orc, torch_dev, small_f32):
    """float32 vectors through k-means, cluster placement and ordered admission:
    answers equal the oracle's bit for bit."""
    a, q, oids, od, oc = small_f32
    n2s, cent = g.cluster_order(a["x"], 12, iterations=3)
    assert np.array_equal(np.sort(n2s), np.arange(len(a["x"]), dtype=np.uint32))
    ix = g.Index(a["x"], a["graph"], node_to_slot=n2s)
    ix.set_cache(int(0.08 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=5.0, oversub=4)
    ix.set_query_order(cent)
    gi, gd, st = search(torch_dev, ix, q, 10, 128, 8)
    assert_same(gi, gd, oids, od)
    assert st["misses"] > 0
    ix.close()
