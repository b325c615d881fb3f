"""GPU resume queue (mode 3): fill waves queue the lanes parked on the slots
they fill and executor waves run the queued lanes' turns, with nothing on the
host but the proxy and the watchdog.  Every result must equal the CPU oracle
bit for bit, whatever the cache, latency, lane count or placement."""
import numpy as np
import pytest

import paper_2607_04415_amd as g
from workload import WORKLOADS, index_arrays, query_array
from test_gpu_modes import assert_same, search, small, small_f32, torch_dev  # noqa: F401  (fixtures)

pytestmark = pytest.mark.gpu
QUEUE = 3


@pytest.mark.parametrize("frac,latency,vfirst,lanes", [
    (0.10, 0.0, False, 0), (0.10, 20.0, True, 0), (0.30, 5.0, False, 7), (0.05, 0.0, True, 1), (0.10, 0.0, True, 40),
], ids=["c10-l0", "c10-l20-vfirst", "c30-l5-7lanes", "c5-l0-1lane", "c10-l0-40lanes"])
def test_gpu_queue_matches_oracle(torch_dev, small, monkeypatch, frac, latency, vfirst, lanes):
    a, q, oids, od, oc = small
    monkeypatch.setenv("GORIO_WATCHDOG_S", "30")
    ix = g.Index(a["x"], a["graph"], vectors_first=vfirst)
    ix.set_cache(max(int(frac * ix.info["index_bytes"]), 128 * 4096))
    ix.set_backing(latency_us=latency, mode=QUEUE)
    ix.set_scheduler(query_waves=lanes)
    print(f"[gpu queue] frac={frac} latency={latency} vfirst={vfirst} lanes={lanes}", flush=True)
    gi, gd, st = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    assert st["iterations"] == int(oc["iterations"].sum())
    assert st["hits"] + st["misses"] == st["expansions"] + st["evaluations"]
    assert st["misses"] > 0 and st["pages_served"] > 0 and st["parks"] > 0 and st["resumes"] > 0
    ix.close()


def test_gpu_queue_f32_clusters(torch_dev, small_f32, monkeypatch):
    """float32 rows, cluster placement and cluster-ordered admission."""
    a, q, oids, od, oc = small_f32
    monkeypatch.setenv("GORIO_WATCHDOG_S", "30")
    n2s, cent = g.cluster_order(a["x"], 12, iterations=3)
    ix = g.Index(a["x"], a["graph"], node_to_slot=n2s, vectors_first=True)
    ix.set_cache(int(0.08 * ix.info["index_bytes"]))
    ix.set_backing(latency_us=5.0, mode=QUEUE)
    ix.set_query_order(cent)
    print("[gpu queue] f32 clusters", flush=True)
    gi, gd, st = search(torch_dev, ix, q, 10, 128, 8)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    ix.close()


def test_gpu_queue_held_proxy_then_recover(torch_dev, small, monkeypatch):
    """A proxy that never completes: the search ends at the watchdog with
    GORIO_ETIMEOUT (every wave leaves on the abort flag), and the next search
    is normal."""
    a, q, oids, od, _ = small
    ix = g.Index(a["x"], a["graph"])
    ix.set_cache(300 * 4096)
    ix.set_backing(latency_us=0.0, mode=QUEUE)
    monkeypatch.setenv("GORIO_PROXY_HOLD", "1")
    monkeypatch.setenv("GORIO_WATCHDOG_S", "1")
    print("[gpu queue] held proxy", flush=True)
    with pytest.raises(g.GorioError) as e:
        search(torch_dev, ix, q, 10, 32, 4)
    assert e.value.status == g.ETIMEOUT
    monkeypatch.delenv("GORIO_PROXY_HOLD")
    monkeypatch.setenv("GORIO_WATCHDOG_S", "30")
    gi, gd, _ = search(torch_dev, ix, q, 10, 32, 4)
    assert_same(gi, gd, oids, od)
    ix.close()


def test_gpu_queue_1m_bench_configuration(orc, torch_dev, monkeypatch):
    """The 1M uint8 index, 10% cold cache, 0 us, all 10,000 queries, pages
    placed by 512 clusters and queries admitted by cluster, 40 lanes."""
    monkeypatch.setenv("GORIO_WATCHDOG_S", "60")
    w = WORKLOADS["u8-1m-cache10-lat0"]
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)
    n2s, cent = g.cluster_order(a["x"], 512)
    ix = g.Index(a["x"], a["graph"], vectors_first=True, node_to_slot=n2s)
    ix.set_cache(int(w.cache_frac * ix.info["index_bytes"]))
    ix.set_backing(latency_us=w.latency_us, mode=QUEUE)
    ix.set_scheduler(query_waves=40)
    ix.set_query_order(cent)
    print("[gpu queue] 1m bench configuration", flush=True)
    gi, gd, st = search(torch_dev, ix, q, w.k, w.L, w.W)
    e = ix.info["entry"]
    ix.close()
    oids, od, oc, _ = orc.pack(a["x"], a["graph"]).search(q, w.k, w.L, w.W, e, threads=16)
    assert_same(gi, gd, oids, od)
    assert st["expansions"] == int(oc["expansions"].sum())
    hr = st["hits"] / max(1, st["hits"] + st["misses"])
    print(f"[gpu queue 1m] {len(q)} queries, {st['kernel_ms']:.0f} ms, {len(q) / st['kernel_ms'] * 1e3:,.0f} q/s, "
          f"hit rate {hr:.3f}", flush=True)
