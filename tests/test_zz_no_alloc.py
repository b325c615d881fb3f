"""gorio_search_noalloc (the resident search without any allocation) against
gorio_search, called through the C ABI: the same ids and distance bits on two
calls in a row, the second with a smaller batch, so the shared scratch words
left by the first call must not leak into the second."""
import ctypes

import numpy as np
import pytest

import paper_2607_04415_amd as g
from workload import IndexSpec, QuerySpec, index_arrays, query_array

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    torch.cuda.set_device(0)
    return torch


def _noalloc():
    return g.lib().gorio_search_noalloc


def _search(torch, fn, ix, qd, nq, k, L, W, dtype):
    ids = torch.full((nq, k), -7, dtype=torch.int32, device="cuda")
    dists = torch.full((nq, k), -7, dtype=dtype, device="cuda")
    st = g.Stats()
    stream = torch.cuda.current_stream().cuda_stream
    status = fn(ix._h, qd.data_ptr(), nq, k, L, W, ids.data_ptr(), dists.data_ptr(), ctypes.byref(st),
                ctypes.c_void_p(stream))
    assert status == g.OK, g.lib().gorio_last_error().decode()
    torch.cuda.synchronize()
    return ids.cpu().numpy().view(np.uint32), dists.cpu().numpy(), st.as_dict()


@pytest.mark.parametrize("dtype", ["u8", "f32"])
def test_noalloc_matches_search_twice(torch_dev, dtype):
    torch = torch_dev
    spec = (IndexSpec(n=20000, D=128, dtype="u8", clusters=16, sigma=20.0, r_near=16, r_rand=16, seed=71)
            if dtype == "u8" else
            IndexSpec(n=12000, D=96, dtype="f32", clusters=8, sigma=0.05, r_near=32, r_rand=32, seed=72))
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(3000, 73))
    k, L, W = (10, 64, 4) if dtype == "u8" else (10, 128, 8)
    tdt = torch.int32 if dtype == "u8" else torch.float32
    ix = g.Index(a["x"], a["graph"], vectors_first=True)
    qd = torch.from_numpy(q).cuda()
    ref = _search(torch, g.lib().gorio_search, ix, qd, len(q), k, L, W, tdt)
    fn = _noalloc()
    for nq in (len(q), 777):     # the second call is smaller than the first
        ids, dists, st = _search(torch, fn, ix, qd, nq, k, L, W, tdt)
        assert np.array_equal(ids, ref[0][:nq])
        assert np.array_equal(dists.view(np.uint32), ref[1][:nq].view(np.uint32))
        # counters are this call's only (the scratch is cleared per call)
        assert 0 < st["expansions"] <= ref[2]["expansions"]
        if nq == len(q):
            assert st["expansions"] == ref[2]["expansions"]
            assert st["evaluations"] == ref[2]["evaluations"]
    ix.close()


def test_noalloc_rejects(torch_dev):
    torch = torch_dev
    spec = IndexSpec(n=3000, D=128, dtype="u8", clusters=4, sigma=20.0, r_near=8, r_rand=8, seed=74)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(50, 75))
    ix = g.Index(a["x"], a["graph"])
    fn = _noalloc()
    qh = np.ascontiguousarray(q)
    ids = np.empty((50, 10), np.uint32)
    dists = np.empty((50, 10), np.int32)
    # host pointers: rejected (the call would have to stage them)
    assert fn(ix._h, qh.ctypes.data, 50, 10, 32, 4, ids.ctypes.data, dists.ctypes.data, None, None) == g.EINVAL
    qd = torch.from_numpy(q).cuda()
    idd = torch.empty((50, 10), dtype=torch.int32, device="cuda")
    dd = torch.empty((50, 10), dtype=torch.int32, device="cuda")
    assert fn(ix._h, qd.data_ptr(), 50, 10, 300, 4, idd.data_ptr(), dd.data_ptr(), None, None) == g.EINVAL
    # paged indexes are not served by this entry point
    ix.set_cache(64 * 4096)
    assert fn(ix._h, qd.data_ptr(), 50, 10, 32, 4, idd.data_ptr(), dd.data_ptr(), None, None) == g.EUNSUPPORTED
    ix.close()


def test_noalloc_graph_replays(torch_dev):
    """Captured into a HIP graph, gorio_search_noalloc replays the whole
    search each time: every replay gives gorio_search's answers, with eager
    searches (which reuse the same scratch words) between the replays."""
    torch = torch_dev
    spec = IndexSpec(n=20000, D=128, dtype="u8", clusters=16, sigma=20.0, r_near=16, r_rand=16, seed=76)
    a = index_arrays(spec, use_cache=False)
    q = query_array(spec, QuerySpec(2000, 77))
    k, L, W = 10, 64, 4
    nq = len(q)
    ix = g.Index(a["x"], a["graph"], vectors_first=True)
    qd = torch.from_numpy(q).cuda()
    search, fn = g.lib().gorio_search, _noalloc()
    ref_ids, ref_d, _ = _search(torch, search, ix, qd, nq, k, L, W, torch.int32)
    ids = torch.full((nq, k), -7, dtype=torch.int32, device="cuda")
    dists = torch.full((nq, k), -7, dtype=torch.int32, device="cuda")
    # first call on this device outside the capture (it looks the scratch up)
    _search(torch, fn, ix, qd, 100, k, L, W, torch.int32)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        # statistics need a synchronisation: refused under capture
        assert fn(ix._h, qd.data_ptr(), nq, k, L, W, ids.data_ptr(), dists.data_ptr(),
                  ctypes.byref(g.Stats()), s) == g.EINVAL
        # gorio_search keeps a host-side ticket base: refused under capture
        assert search(ix._h, qd.data_ptr(), nq, k, L, W, ids.data_ptr(), dists.data_ptr(), None, s) \
            == g.EUNSUPPORTED
        status = fn(ix._h, qd.data_ptr(), nq, k, L, W, ids.data_ptr(), dists.data_ptr(), None, s)
    assert status == g.OK, g.lib().gorio_last_error().decode()
    torch.cuda.synchronize()
    for rep in range(3):
        ids.fill_(-7)
        dists.fill_(-7)
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(ids.cpu().numpy().view(np.uint32), ref_ids), rep
        assert np.array_equal(dists.cpu().numpy(), ref_d), rep
        # eager work on the same index and scratch between replays
        e_ids, e_d, _ = _search(torch, fn, ix, qd, 300 + 200 * rep, k, L, W, torch.int32)
        assert np.array_equal(e_ids, ref_ids[:300 + 200 * rep])
        e_ids, e_d, _ = _search(torch, search, ix, qd, 500, k, L, W, torch.int32)
        assert np.array_equal(e_ids, ref_ids[:500])
    del graph
    ix.close()
