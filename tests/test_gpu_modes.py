"""GPU parity of the scheduling modes and scheduler shapes of the paged search.

Host-scheduled lanes (mode 2: a host thread owns the query lanes and decides
which run, as their pages are filled; a persistent executor launch runs the
turns it hands over through a ring, or a launch per round runs them),
the blocking and split-phase modes at an equal number of query waves
(gorio_set_scheduler), and the full 10M x 96-d float32 configuration: every
result must equal the CPU oracle bit for bit (float32 distances compared as
uint32 bit patterns), whatever the mode.
"""
import os

import numpy as np
import pytest

import paper_2607_04415_amd as g
from workload import IndexSpec, QuerySpec, WORKLOADS, index_arrays, query_array

pytestmark = pytest.mark.gpu

SPEC = IndexSpec(n=20000, D=128, dtype="u8", clusters=8, sigma=20.0, r_near=16, r_rand=16, seed=41)
F32_SPEC = IndexSpec(n=12000, D=96, dtype="f32", clusters=8, sigma=0.05, r_near=32, r_rand=32, seed=45)
HOST = 2


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    torch.cuda.set_device(0)
    return torch


def oracle_answers(orc, a, q, k, L, W):
    e = orc.medoid(a["x"])
    return orc.pack(a["x"], a["graph"]).search(q, k, L, W, e, threads=16)


@pytest.fixture(scope="module")
def small(orc):
    a = index_arrays(SPEC, use_cache=False)
    q = query_array(SPEC, QuerySpec(400, 42))
    oids, od, oc, _ = oracle_answers(orc, a, q, 10, 32, 4)
    return a, q, oids, od, oc


@pytest.fixture(scope="module")
def small_f32(orc):
    a = index_arrays(F32_SPEC, use_cache=False)
    q = query_array(F32_SPEC, QuerySpec(300, 46))
    oids, od, oc, _ = oracle_answers(orc, a, q, 10, 128, 8)
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


# --------------------------------------------------------------------------- #
# host-scheduled lanes
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("frac,latency,vfirst,lanes,passes", [
    (0.10, 0.0, False, 0, None), (0.10, 20.0, True, 0, None), (0.30, 5.0, False, 7, "3"), (0.05, 0.0, True, 1, None),
    (0.10, 0.0, True, 0, "0"),
], ids=["c10-l0", "c10-l20-vfirst", "c30-l5-7lanes-3passes", "c5-l0-1lane", "c10-l0-unbounded-turns"])
def test_host_rounds_match_oracle(torch_dev, small, monkeypatch, frac, latency, vfirst, lanes, passes):
    a, q, oids, od, oc = small
    if passes is not None:
        monkeypatch.setenv("GORIO_TURN_PASSES", passes)
    ix = g.Index(a["x"], a["graph"], vectors_first=vfirst)
    ix.set_cache(max(int(frac * ix.info["index_bytes"]), 128 * 4096))
    ix.set_backing(latency_us=latency, mode=HOST)
    ix.set_scheduler(query_waves=lanes)
    print(f"[host rounds] frac={frac} latency={latency} vfirst={vfirst} lanes={lanes}", flush=True)
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    assert st["iterations"] == int(oc["iterations"].sum())
    assert st["hits"] + st["misses"] == st["expansions"] + st["evaluations"]
    assert st["misses"] > 0 and st["pages_served"] > 0 and st["parks"] > 0
    ix.close()


@pytest.mark.parametrize("flights,lanes,passes", [("2", 0, None), ("4", 0, None), ("8", 12, "0")])
def test_host_rounds_launch_per_round(torch_dev, small, monkeypatch, flights, lanes, passes):
    """Host-scheduled lanes run by a launch per round (instead of the
    persistent executor), with one or several round kernels in flight on
    streams of their own, lanes retired one by one as their reports arrive and
    launched again on whichever stream is free: the answers and counts stay
    the oracle's."""
    a, q, oids, od, oc = small
    monkeypatch.setenv("GORIO_HOST_EXECUTOR", "0")
    monkeypatch.setenv("GORIO_ROUND_FLIGHTS", flights)
    if passes is not None:
        monkeypatch.setenv("GORIO_TURN_PASSES", passes)
    ix = g.Index(a["x"], a["graph"], vectors_first=True)
    ix.set_cache(int(0.10 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=5.0, mode=HOST)
    ix.set_scheduler(query_waves=lanes)
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    assert st["iterations"] == int(oc["iterations"].sum())
    ix.close()


def test_host_rounds_f32_clusters(orc, torch_dev, small_f32):
    """float32 rows, cluster placement and cluster-ordered admission, host rounds."""
    a, q, oids, od, oc = small_f32
    n2s, cent = g.cluster_order(a["x"], 12, iterations=3)
    ix = g.Index(a["x"], a["graph"], node_to_slot=n2s, vectors_first=True)
    ix.set_cache(int(0.08 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=5.0, mode=HOST)
    ix.set_query_order(cent)
    gi, gd, st = search(torch_dev, ix, q, 10, 128, 8)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    ix.close()


def test_host_rounds_held_proxy_then_recover(torch_dev, small, monkeypatch):
    """A proxy that never completes: the host-scheduled search ends at the
    watchdog with GORIO_ETIMEOUT, and the next search is normal."""
    a, q, oids, od, _ = small
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(300 * 4096)
    ix.set_backing(latency_us=0.0, mode=HOST)
    monkeypatch.setenv("GORIO_PROXY_HOLD", "1")
    monkeypatch.setenv("GORIO_WATCHDOG_S", "1")
    with pytest.raises(g.GorioError) as e:
        search(torch_dev, ix, q, 10, 32, 4)
    assert e.value.status == g.ETIMEOUT
    monkeypatch.delenv("GORIO_PROXY_HOLD")
    monkeypatch.delenv("GORIO_WATCHDOG_S")
    gi, gd, _ = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    ix.close()


@pytest.mark.parametrize("executor", ["1", "0"], ids=["executor", "launch-per-round"])
def test_host_rounds_with_many_streams_alive(torch_dev, small, monkeypatch, executor):
    """Host-scheduled lanes while the process holds many more streams than
    the device has hardware queues, so streams share queues (and work on a
    shared queue may run one item after another).  No kernel of the mode waits
    for another stream's work (the executor is one launch; with a launch per
    round the fill kernel leaves after a budget and is launched again), so the
    search finishes, exactly."""
    torch = torch_dev
    a, q, oids, od, oc = small
    monkeypatch.setenv("GORIO_HOST_EXECUTOR", executor)
    streams = [torch.cuda.Stream() for _ in range(12)]
    keep = []
    for s in streams:   # use every stream once, so each holds its queue
        with torch.cuda.stream(s):
            keep.append(torch.ones(1024, device="cuda") * 2)
    torch.cuda.synchronize()
    monkeypatch.setenv("GORIO_WATCHDOG_S", "60")
    ix = g.Index(a["x"], a["graph"], vectors_first=True)
    ix.set_cache(int(0.10 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=5.0, mode=HOST)
    qd = torch.from_numpy(np.ascontiguousarray(q)).cuda()
    torch.cuda.synchronize()          # the queries are in place before another stream reads them
    for s in (streams[3], streams[7]):
        ids, dists, st = ix.search(qd, 10, 32, 4, stream=s.cuda_stream)
        torch.cuda.synchronize()
        assert_same(ids.cpu().numpy().view(np.uint32), dists.cpu().numpy(), oids, od)
        assert st["expansions"] == int(oc["expansions"].sum())
        assert st["pages_served"] > 0
    ix.close()
    assert all(float(k.sum()) == 2048.0 for k in keep)


def test_host_rounds_1m_bench_configuration(orc, torch_dev):
    """The 1M uint8 index, 10% cold cache, 0 us, all 10,000 queries, in the
    benchmark's launch configuration for the host-scheduled leg (40 lanes run
    by the persistent executor, vectors-first pages placed by 512 clusters,
    queries admitted by cluster)."""
    w = WORKLOADS["u8-1m-cache10-lat0"]
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)
    n2s, cent = g.cluster_order(a["x"], 512)
    ix = g.Index(a["x"], a["graph"], vectors_first=True, node_to_slot=n2s)
    ix.set_cache(int(w.cache_frac * ix.info["index_bytes"]))
    ix.set_backing(latency_us=w.latency_us, mode=HOST)
    ix.set_scheduler(query_waves=40)
    ix.set_query_order(cent)
    gi, gd, st = search(torch_dev, ix, q, w.k, w.L, w.W)
    e = ix.info["entry"]
    ix.close()
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, w.k, w.L, w.W, e, threads=16)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    hr = st["hits"] / max(1, st["hits"] + st["misses"])
    print(f"[host rounds 1m] {len(q)} queries, {st['kernel_ms']:.0f} ms, hit rate {hr:.3f}", flush=True)


# --------------------------------------------------------------------------- #
# scheduler shape: equal query waves for blocking and split-phase
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("mode,oversub,waves,pending", [
    (1, 1, 3, 32), (0, 4, 3, 8), (0, 4, 3, 32), (1, 1, 2, 4), (0, 2, 0, 1),
], ids=["blocking-3w", "split-3w-p8", "split-3w-p32", "blocking-2w-p4", "split-p1"])
def test_scheduler_shape_same_answers(torch_dev, small, mode, oversub, waves, pending):
    a, q, oids, od, oc = small
    ix = g.Index(a["x"], a["graph"], vectors_first=True)
    ix.set_cache(int(0.10 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=20.0, oversub=oversub, mode=mode)
    ix.set_scheduler(query_waves=waves, max_pending=pending)
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    ix.close()


def test_scheduler_rejects(torch_dev, small):
    a, q, _, _, _ = small
    ix = g.Index(a["x"], a["graph"])
    for kw in (dict(query_waves=65537), dict(max_pending=257)):
        with pytest.raises(g.GorioError) as e:
            ix.set_scheduler(**kw)
        assert e.value.status == g.EINVAL
    with pytest.raises(g.GorioError) as e:
        ix.set_backing(mode=4)                           # modes are 0..3
    assert e.value.status == g.EINVAL
    ix.close()


# --------------------------------------------------------------------------- #
# the 10M x 96-d float32 configuration at its full query count
# --------------------------------------------------------------------------- #
F32_10M = WORKLOADS["f32-10m-cache5-lat20"]


@pytest.mark.timeout(1200)
@pytest.mark.skipif(os.environ.get("GORIO_SKIP_BIG") == "1",
                    reason="GORIO_SKIP_BIG=1: the 10M float32 index takes minutes to generate and check")
def test_workload_f32_10m_full(orc, torch_dev):
    """All 100,000 queries of the 10M x 96-d float32 configuration, in the
    benchmark's launch configurations: the HBM-resident search (vectors-first
    pages) and the paged search (5% cold cache, 20 us per request, 60 query
    waves of one query, pages placed by 1024 clusters, queries admitted by
    cluster).  Both equal the oracle element by element: ids and distance bits,
    after the 1e-5 relative / 0.999 id-overlap acceptance bound."""
    w = F32_10M
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)
    assert len(q) == 100_000
    ix = g.Index(a["x"], a["graph"], vectors_first=True)
    e = ix.info["entry"]
    ri, rd, rst = search(torch_dev, ix, q, w.k, w.L, w.W)
    ix.close()
    print(f"[f32 10m full] resident search done ({rst['kernel_ms']:.1f} ms)", flush=True)
    n2s, cent = g.cluster_order(a["x"], 1024)
    px = g.Index(a["x"], a["graph"], vectors_first=True, node_to_slot=n2s)
    px.set_cache(int(w.cache_frac * px.info["index_bytes"]))
    px.set_backing(latency_us=w.latency_us, oversub=1)
    px.set_scheduler(query_waves=60)
    px.set_query_order(cent)
    gi, gd, st = search(torch_dev, px, q, w.k, w.L, w.W)
    px.close()
    print(f"[f32 10m full] resident {rst['kernel_ms']:.1f} ms, paged {st['kernel_ms']:.0f} ms, "
          f"hit rate {st['hits'] / max(1, st['hits'] + st['misses']):.3f}", flush=True)
    assert e == orc.medoid(a["x"])
    packed = orc.pack(a["x"], a["graph"])
    print("[f32 10m full] oracle pages packed", flush=True)
    oids, od, oc = [], [], []
    for lo in range(0, len(q), 10_000):     # in slices, so progress shows
        i_, d_, c_, _ = packed.search(q[lo:lo + 10_000], w.k, w.L, w.W, e, threads=16)
        oids.append(i_), od.append(d_), oc.append(c_)
        print(f"[f32 10m full] oracle {lo + len(i_):,} queries", flush=True)
    oids, od, oc = np.concatenate(oids), np.concatenate(od), np.concatenate(oc)
    print("[f32 10m full] oracle done", flush=True)
    from test_gpu_parity import f32_acceptance
    for name, (xi, xd, xs) in (("resident", (ri, rd, rst)), ("paged", (gi, gd, st))):
        f32_acceptance(xi, xd, oids, od)
        assert_same(xi, xd, oids, od)
        assert xs["expansions"] == int(oc["expansions"].sum()), name
        assert xs["iterations"] == int(oc["iterations"].sum()), name
