"""Benchmark: batched paged graph beam search on one MI355X.

One step = one gorio_search over the whole query batch of the workload (all
steps of the search path).  Default workload: 1,000,000 x 128-d uint8 vectors,
R = 64, 388-B records, 10 per 4 KB page, 10,000 queries, k = 10, L = 64, W = 4,
every page resident in HBM.

Prints one JSON line.  `value` is queries per second over the timed steps
(inputs already resident in HBM).  `roofline` prices the search kernel's
algorithmic bytes (expansions x (4 + 4R) + first-time evaluations x vector
bytes) against its average duration, measured with HIP events on the launch
stream; `achieved_hbm_gbs` is the HBM traffic rocprofv3 counted for the same
kernel (committed counter summary) over that duration.  `cpu_baseline` times
the CPU oracle.  The same line carries the other configurations: the small
uint8 index and the 10M x 96-d float32 index resident in HBM
(`resident_legs`), and the paged legs (`paged`: cold 10% / 5% caches behind
the host proxy, the blocking and host-scheduled modes, an equal-wave
split-phase vs blocking comparison over injected latencies).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import subprocess
import sys
import time
from pathlib import Path

import numpy as np

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

METRIC = "queries/sec at k=10 (oracle-exact) + achieved HBM GB/s and miss-service GB/s"
HBM_PEAK_GBS = 8000.0
# page layouts (both put the same nodes in the same 4 KB pages; see include/gorio.h)
LAYOUTS = ("vectors-first", "contiguous")
PROFILES = ROOT / "profiles"
KERNEL_SOURCES = ["paper_2607_04415_amd/csrc/search_resident.hpp", "paper_2607_04415_amd/csrc/frontier.hpp",
                  "paper_2607_04415_amd/csrc/metric.hpp", "paper_2607_04415_amd/csrc/launch.hpp",
                  "paper_2607_04415_amd/csrc/common.hpp", "paper_2607_04415_amd/csrc/wave.hpp"]
MODES = {0: "split-phase", 1: "blocking", 2: "host-scheduled", 3: "gpu resume queue"}
# Scheduler shapes of the paged legs (oversub = query slots per wave, query_waves; 0 = the
# library's default, which runs as many queries as the cache's pins allow).  When the host
# link is the bound, fewer queries in flight keep the link full and share the cache better
# (sweeps on the full query counts: 1M index, 10% cache, 0 us, 256 clusters: 20 / 30 / 40
# waves x 1 slot 6,754 / 7,451 / 7,392 queries/s; 512 clusters: 30 x 1 7,597 against 6,260
# for the default 156 queries in 39 waves x 4 slots; 10M float32, 5% cache, 512 clusters:
# 40 / 60 / 80 waves x 1 slot 3,285 / 3,426 / 3,386, the default 1,302 queries far less).
# The 100k-query 20 us configuration asks for 4 query slots per wave: 30 waves gave 8,512
# against 8,351 for the default 39.
SHAPE_C3 = {"oversub": 1, "query_waves": 30}
# host-scheduled lanes (persistent executor, turns until a lane parks): 30 / 40 / 50 / 60 /
# 100 / 156 (the default) lanes gave 7.0k / 7.25k / 7.2k / 7.05k / 6.6k / 6.0k queries/s
SHAPE_HOST = {"query_waves": 40}
# GPU resume queue (fill waves queue the lanes parked on the pages they fill, executor
# waves run them): 30 / 40 / 60 lanes gave 7.0k / 7.2k / 7.1k queries/s (20 / 100 / 156,
# the default, 6.2k / 6.6k / 6.0k before resumed lanes withdrew their other waits)
SHAPE_QUEUE = {"query_waves": 40}
SHAPE_C4 = {"oversub": 4, "query_waves": 30}
SHAPE_C5 = {"oversub": 1, "query_waves": 60}
# The paper's own figures (Table 2: 10,000 SIFT1M queries over NVMe-oF on one NVIDIA L40S,
# ConnectX-6 200 Gb/s InfiniBand, a remote NVMe SSD; Table 1).  Context, not targets: a
# different machine, transport and dataset.
PAPER_CONTEXT = {
    "hardware": "NVIDIA L40S 48 GB, Xeon Silver 4316, ConnectX-6 200 Gb/s InfiniBand, remote NVMe SSD over NVMe-oF",
    "workload": "SIFT1M DiskANN-style graph, 10,000 queries, top-10",
    "qps": {"G-Gust (host scheduler over GORIO's backend)": 10058, "GustANN-SPDK": 7680,
            "G-ABaM (GPU split-phase scheduler)": 5650, "G-BaM (blocking)": 1155, "GDS": 83},
    "speedups": {"G-Gust vs GustANN-SPDK": 1.31, "G-ABaM vs G-BaM": 4.89},
}
T_START = time.perf_counter()


def log(msg):
    print(f"[bench {time.perf_counter() - T_START:6.1f}s] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        h.update((ROOT / p).read_bytes())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, layout: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source and page layout; else None."""
    f = PROFILES / f"traffic_{workload}.json"
    if not f.exists():
        return None
    try:
        t = json.loads(f.read_text())
    except ValueError:
        return None
    if t.get("kernel_source_hash") != kernel_source_hash() or t.get("layout") != layout:
        return None
    return t.get("hbm_bytes_per_launch")


def oracle_threads() -> tuple[int, int]:
    """(T, nproc): threads for the CPU oracle and the CPUs this process may run
    on.  T is nproc, capped at the host's per-GPU CPU share (OMP_NUM_THREADS,
    else 16)."""
    nproc = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    share = int(os.environ.get("OMP_NUM_THREADS", "16") or 16)
    return max(1, min(nproc, share)), nproc


def cpu_baseline(a, q, w, gpu_ids, gpu_dists, sample_nq: int, one_thread_nq: int, packed=None):
    """Time the CPU oracle on the first `sample_nq` queries with T threads on
    disjoint shards, and with one thread on the first `one_thread_nq`; also
    check the GPU answers on the T-thread sample."""
    from oracle import load
    orc = load()
    t0 = time.perf_counter()
    if packed is None:
        packed = orc.pack(a["x"], a["graph"])
    entry = orc.medoid(a["x"])
    prep = time.perf_counter() - t0
    threads, nproc = oracle_threads()
    qs = q[:sample_nq]
    t0 = time.perf_counter()
    oids, od, oc, _ = packed.search(qs, w.k, w.L, w.W, entry, threads=threads)
    dt = time.perf_counter() - t0
    exact = bool(np.array_equal(oids, gpu_ids[:sample_nq])
                 and np.array_equal(od.view(np.uint32), gpu_dists[:sample_nq].view(np.uint32)))
    one = None
    if one_thread_nq > 0:
        t0 = time.perf_counter()
        packed.search(q[:one_thread_nq], w.k, w.L, w.W, entry, threads=1)
        dt1 = time.perf_counter() - t0
        one = {"value": round(one_thread_nq / dt1, 1), "unit": "queries/s",
               "sample": f"first {one_thread_nq} queries, 1 thread, {dt1:.2f} s"}
    counts = {"queries": len(qs), "evaluations": int(oc["evaluations"].sum()),
              "expansions": int(oc["expansions"].sum()), "iterations": int(oc["iterations"].sum())}
    base = {
        "value": round(sample_nq / dt, 1), "unit": "queries/s", "cores": threads, "kind": "oracle",
        "sample": f"first {sample_nq} of {len(q)} queries of the same workload, {threads} threads on "
                  f"disjoint query shards, {dt:.2f} s wall (page packing and medoid {prep:.1f} s, not timed)",
        "nproc": nproc, "one_thread": one,
    }
    return base, exact, entry, counts, (oids, od), packed


def recall_at_k(x: np.ndarray, q: np.ndarray, ids: np.ndarray, k: int, sample: int) -> dict:
    """Recall@k of the search answers against exact top-k (squared L2, ties by
    id) on the first `sample` queries; informational (the paper reports QPS
    with Recall@10).  Distances are formed in float64: exact integers for uint8
    data; for float32 data near-ties may order differently from float32 sums."""
    qs, got = q[:sample], ids[:sample]
    xf = x.astype(np.float64)
    xx = (xf * xf).sum(1)
    hits = 0
    for i in range(0, len(qs), 50):
        qf = qs[i:i + 50].astype(np.float64)
        d = (qf * qf).sum(1)[:, None] + xx[None, :] - 2.0 * (qf @ xf.T)
        if x.dtype == np.uint8:
            d = np.rint(d).astype(np.int64)
        for j in range(len(qf)):
            cand = np.argpartition(d[j], k)[:k + 64]
            exact = cand[np.lexsort((cand, d[j][cand]))][:k]
            hits += len(np.intersect1d(exact, got[i + j][:k]))
    return {"value": round(hits / (len(qs) * k), 4), "k": k, "queries": len(qs)}


def gather_ceiling(n: int, rpp: int, page_bytes: int, vec_stride: int):
    """Random 128-byte vector reads from the same page geometry with no search
    around them (paper_2607_04415_amd/microbench/gather_ceiling.hip): the
    practical ceiling of the resident kernel's dominant traffic."""
    from paper_2607_04415_amd import _build
    exe = _build.GATHER_CEILING
    if not exe.exists():
        return None
    r = subprocess.run([str(exe), str(n), str(rpp), str(page_bytes), str(vec_stride)],
                       capture_output=True, text=True, timeout=120)
    if r.returncode != 0:
        log(f"gather ceiling probe failed: {r.stderr.strip()}")
        return None
    d = json.loads(r.stdout.strip().splitlines()[-1])
    best = max(d[k]["gbs"] for k in d if k.startswith("rounds_"))
    return {"gbs": best, "vectors": d["vectors"], "waves": d["waves"],
            "depths_gbs": {k: d[k]["gbs"] for k in d if k.startswith("rounds_")}}


def cluster_count(arg: int, nq: int) -> int:
    """k-means clusters for a paged leg on the 1M index: `arg` if positive, none
    if 0, else 512 (best of 128 / 256 / 512 / 768 / 1024 on the 10k-query leg,
    and of 512 / 768 / 1024 on the 100k-query leg, with the current cache
    policy).  Queries are admitted cluster by cluster."""
    if arg >= 0:
        return arg
    return 512


def host_link_peak_gbs(torch) -> float:
    """Pinned host -> HBM copy bandwidth (256 MiB, best of 5), the host-link ceiling."""
    src = torch.empty(1 << 28, dtype=torch.uint8).pin_memory()
    dst = torch.empty(1 << 28, dtype=torch.uint8, device="cuda")
    best = 0.0
    for _ in range(5):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src, non_blocking=True)
        b.record()
        torch.cuda.synchronize()
        best = max(best, src.numel() / (a.elapsed_time(b) * 1e-3) / 1e9)
    return best


def algorithmic_bytes(st: dict, R: int, vec_bytes: int, oracle_evals=None):
    """(bytes, source): expansions x (4 + 4R) + first-time evaluations x vector
    bytes.  First-time evaluations are the oracle's |V| when it ran on the whole
    batch; otherwise the GPU's evaluations minus those its visited filter could
    not record (a lower bound: an unrecorded evaluation may still be a first)."""
    if oracle_evals is not None:
        return st["expansions"] * (4 + 4 * R) + oracle_evals * vec_bytes, "oracle"
    return st["expansions"] * (4 + 4 * R) + (st["evaluations"] - st["reevaluations"]) * vec_bytes, \
        "gpu lower bound (evaluations minus unrecorded ones)"


def resident_leg(torch, g, a, q, w, layout: str, steps: int, warmup: int):
    """Build the index in `layout`, run the warm-up and the timed steps.

    Timed steps are issued back to back on the stream, as a serving loop would:
    no host round trip per batch (the call returns once the search is queued).
    HIP events recorded on the same stream around each call give every launch's
    duration; the counters come from one more call after the timed region."""
    ix = g.Index(a["x"], a["graph"], vectors_first=layout == "vectors-first")
    info = ix.info
    nq = len(q)
    qd = torch.from_numpy(q).cuda()
    ids = torch.empty((nq, w.k), dtype=torch.int32, device="cuda")
    dists = torch.empty((nq, w.k), dtype=torch.int32 if q.dtype == np.uint8 else torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    for _ in range(warmup):
        ix.search_into(qd, nq, w.k, w.L, w.W, ids, dists, stream=stream)
    cur = torch.cuda.current_stream()
    events = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        ix.search_into(qd, nq, w.k, w.L, w.W, ids, dists, stream=stream, stats=False)
        e1.record(cur)
        events.append((e0, e1))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kernel_ms = [x.elapsed_time(y) for x, y in events]
    st = ix.search_into(qd, nq, w.k, w.L, w.W, ids, dists, stream=stream)
    ix.close()
    del qd
    log(f"{w.name} {layout}: {steps} steps: {elapsed * 1e3 / steps:.3f} ms/step, {nq * steps / elapsed:,.0f} queries/s")
    return {"info": info, "elapsed": elapsed, "kernel_ms": kernel_ms, "stats": st,
            "ids": ids.cpu().numpy().view(np.uint32), "dists": dists.cpu().numpy()}


def host_buffer_leg(g, a, q, w, layout: str, steps: int, ref_ids, ref_dists) -> dict:
    """The same search with queries, ids and dists in pageable host memory: each
    call stages the queries into HBM and the answers back over the host link and
    returns when they are there.  A rate that includes the link, reported beside
    the HBM-resident one, never as it."""
    ix = g.Index(a["x"], a["graph"], vectors_first=layout == "vectors-first")
    nq = len(q)
    qh = np.ascontiguousarray(q)
    ids = np.empty((nq, w.k), np.uint32)
    dists = np.empty((nq, w.k), np.int32 if q.dtype == np.uint8 else np.float32)
    ix.search_into(qh, nq, w.k, w.L, w.W, ids, dists, stats=False)
    t0 = time.perf_counter()
    for _ in range(steps):
        ix.search_into(qh, nq, w.k, w.L, w.W, ids, dists, stats=False)
    elapsed = time.perf_counter() - t0
    ix.close()
    out = {"value": round(nq * steps / elapsed, 1), "unit": "queries/s", "steps": steps,
           "ms_per_step": round(elapsed * 1e3 / steps, 4),
           "bytes_per_step": {"queries_in": int(qh.nbytes), "answers_out": int(ids.nbytes + dists.nbytes)},
           "same_answers": bool(np.array_equal(ids, ref_ids) and np.array_equal(dists, ref_dists))}
    log(f"{w.name} with host buffers: {out['ms_per_step']:.3f} ms/step, {out['value']:,.0f} queries/s")
    return out


def roofline_of(res: dict, w, R: int, oracle_evals, traffic, kernel: str) -> dict:
    st = res["stats"]
    alg, src = algorithmic_bytes(st, R, w.index.vec_bytes, oracle_evals)
    kms = float(np.mean(res["kernel_ms"]))
    achieved = alg / (kms * 1e-3) / 1e9
    r = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
         "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": kernel,
         "kernel_ms_avg": round(kms, 4), "algorithmic_bytes_per_launch": int(alg), "algorithmic_counts": src}
    if src != "oracle":   # the range the unrecorded evaluations leave open
        hi = st["expansions"] * (4 + 4 * R) + st["evaluations"] * w.index.vec_bytes
        r["algorithmic_upper_gbs"] = round(hi / (kms * 1e-3) / 1e9, 1)
    if traffic:
        r["traffic_gbs"] = round(traffic / (kms * 1e-3) / 1e9, 1)
        r["traffic_frac"] = round(traffic / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    return r


def paged_leg(torch, g, a, w, nq_sample: int, resident_qps: float, mode: int = 0,
              vectors_first: bool = True, repeats: int = 5, clusters=None, warmup_nq: int = 2000,
              query_waves: int = 0, max_pending: int = 0, latency_us=None, oversub=None, label=None):
    """Cold-cache paged searches over the first nq_sample queries of workload w:
    one untimed warm-up search on the first warmup_nq queries, then `repeats`
    timed runs, each from a cache that set_cache has just emptied; the figures
    are the median run's.  clusters = (node_to_slot, centroids): pages placed
    cluster by cluster and queries admitted cluster by cluster."""
    from workload import query_array
    q = query_array(w.index, w.queries)[:nq_sample]
    lat = w.latency_us if latency_us is None else latency_us
    ovs = (w.oversub if oversub is None else oversub) if mode == 0 else 1
    ix = g.Index(a["x"], a["graph"], vectors_first=vectors_first,
                 node_to_slot=None if clusters is None else clusters[0])
    if clusters is not None:
        ix.set_query_order(clusters[1])
    qd = torch.from_numpy(q).cuda()
    ids = torch.empty((len(q), w.k), dtype=torch.int32, device="cuda")
    dists = torch.empty((len(q), w.k), dtype=torch.int32 if q.dtype == np.uint8 else torch.float32,
                        device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def configure():
        ix.set_cache(int(w.cache_frac * ix.info["index_bytes"]))      # empty cache
        ix.set_backing(latency_us=lat, oversub=ovs, mode=mode)
        ix.set_scheduler(query_waves=query_waves, max_pending=max_pending)

    configure()
    wn = min(warmup_nq, len(q))
    ix.search_into(qd[:wn], wn, w.k, w.L, w.W, ids[:wn], dists[:wn], stream=stream)
    runs = []
    for _ in range(max(1, repeats)):
        configure()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st = ix.search_into(qd, len(q), w.k, w.L, w.W, ids, dists, stream=stream)
        torch.cuda.synchronize()
        runs.append((time.perf_counter() - t0, st))
    order = sorted(range(len(runs)), key=lambda i: runs[i][0])
    wall, st = runs[order[len(runs) // 2]]
    ms = st["kernel_ms"]
    acc = st["hits"] + st["misses"]
    out = {"workload": w.name, "queries": len(q), "mode": MODES[mode], "label": label or MODES[mode],
           "placement": "identity" if clusters is None else f"clusters ({len(clusters[1])}, queries by cluster)",
           "cache_slots": ix.info["cache_slots"], "latency_us": lat, "oversub": ovs,
           "query_waves": query_waves or "default", "max_pending": max_pending or 32,
           "warmup_queries": wn, "runs": len(runs),
           "qps": round(len(q) / wall, 1), "qps_runs": [round(len(q) / r[0], 1) for r in runs],
           "kernel_ms": round(ms, 2),
           "hit_rate": round(st["hits"] / max(1, acc), 4),
           "pages_served": st["pages_served"],
           "link_mb_per_query": round(st["bytes_served"] / len(q) / 1e6, 3),
           "miss_service_gbs": round(st["bytes_served"] / (ms * 1e-3) / 1e9, 2),
           "parks": st["parks"], "resumes": st["resumes"], "proxy_peak": st["proxy_peak"],
           "vs_resident_qps": round(len(q) / wall / resident_qps, 5) if resident_qps else None}
    ix.close()
    return out, ids.cpu().numpy().view(np.uint32), dists.cpu().numpy(), q


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="u8-1m-hbm")
    ap.add_argument("--max-queries", type=int, default=0,
                    help="time only the first N queries of the workload (profiling of small batches; 0 = all)")
    ap.add_argument("--layout", choices=LAYOUTS, default="vectors-first",
                    help="page layout of the timed index (the other one is timed too and reported)")
    ap.add_argument("--no-other-layout", action="store_true", help="do not time the other page layout")
    ap.add_argument("--no-host-buffers", action="store_true",
                    help="do not time the search with queries and answers in host memory")
    ap.add_argument("--cpu-sample", type=int, default=10000)
    ap.add_argument("--one-thread-sample", type=int, default=2000,
                    help="queries the 1-thread oracle baseline runs (0 = skip)")
    ap.add_argument("--recall-sample", type=int, default=100,
                    help="queries whose recall@k against exact top-k is reported (0 = skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gather-ceiling", action="store_true",
                    help="skip the random-gather ceiling probe (microbench/gather_ceiling)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (counter calibration)")
    ap.add_argument("--no-small", action="store_true", help="skip the 10k-vector uint8 leg")
    ap.add_argument("--paged-sample", type=int, default=-1,
                    help="queries of each 1M paged configuration to run (-1 = its full query count, "
                         "0 = skip the paged legs)")
    ap.add_argument("--paged-clusters", type=int, default=-1,
                    help="1M paged legs: k-means clusters for page placement and query admission "
                         "(0 = off, -1 = 512)")
    ap.add_argument("--paged-repeats", type=int, default=5,
                    help="cold-cache runs per paged leg of up to 20k queries (the median is reported)")
    ap.add_argument("--large-repeats", type=int, default=3,
                    help="cold-cache runs per paged leg of more than 20k queries")
    ap.add_argument("--ablation-sample", type=int, default=5000,
                    help="queries of the equal-wave split-phase vs blocking comparison (0 = skip)")
    ap.add_argument("--ablation-latencies", default="0,20,200",
                    help="injected latencies (us) of that comparison")
    ap.add_argument("--f32-sample", type=int, default=-1,
                    help="queries of the 10M x 96-d float32 legs (-1 = all 100,000; 0 = skip)")
    ap.add_argument("--no-f32-paged", action="store_true", help="run the float32 resident leg only")
    ap.add_argument("--f32-clusters", type=int, default=1024,
                    help="k-means clusters of the float32 paged leg (512 / 1024 / 2048 / 4096 gave "
                         "3,426 / 4,284 / 4,112 / 3,416 queries/s)")
    ap.add_argument("--f32-cpu-sample", type=int, default=2000,
                    help="float32 queries the oracle runs (baseline and the GPU answers' check)")
    ap.add_argument("--budget-s", type=float, default=500.0,
                    help="legs that would end past this many seconds are skipped and listed")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only (asked for {args.gpus}); "
              "the search shards by query across GPUs but no multi-GPU path is built.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_04415_amd as g
    from workload import WORKLOADS, index_arrays, index_cached, query_array

    if not g.LIB_PATH.exists():
        raise SystemExit("libgorio.so is not built: run python __graft_entry__.py build")
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        # A plain copy kernel of known size: 1 GiB read + 1 GiB written per launch.
        src = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": src.numel() * 4, "launches": 5}), flush=True)
        return
    skipped = []

    def fits(name: str, est_s: float) -> bool:
        if time.perf_counter() - T_START + est_s <= args.budget_s:
            return True
        skipped.append({"leg": name, "estimated_s": est_s,
                        "at_s": round(time.perf_counter() - T_START, 1)})
        log(f"skipping {name}: {est_s:.0f} s would pass the {args.budget_s:.0f} s budget")
        return False

    # ------------------------------------------------------------------ main
    w = WORKLOADS[args.workload]
    log(f"workload {w.name}: {w.description}")
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)
    if args.max_queries > 0:
        q = q[:args.max_queries]
    log("inputs ready")
    nq = len(q)
    main_res = resident_leg(torch, g, a, q, w, args.layout, args.steps, args.warmup)
    info, st = main_res["info"], main_res["stats"]
    qps = nq * args.steps / main_res["elapsed"]
    ms_per_step = main_res["elapsed"] * 1e3 / args.steps
    gi, gd = main_res["ids"], main_res["dists"]
    other = None
    if not args.no_other_layout:
        o_layout = [x for x in LAYOUTS if x != args.layout][0]
        o = resident_leg(torch, g, a, q, w, o_layout, args.steps, args.warmup)
        other = {"layout": o_layout, "value": round(nq * args.steps / o["elapsed"], 1),
                 "ms_per_step": round(o["elapsed"] * 1e3 / args.steps, 4),
                 "kernel_ms_avg": round(float(np.mean(o["kernel_ms"])), 4),
                 "same_answers": bool(np.array_equal(o["ids"], gi) and np.array_equal(o["dists"], gd))}

    host_buffers = None
    if not args.no_host_buffers:
        host_buffers = host_buffer_leg(g, a, q, w, args.layout, args.steps, gi, gd)

    cpu = exact = ocounts = packed_main = None
    if not args.no_cpu_baseline:
        cpu, exact, entry, ocounts, _, packed_main = cpu_baseline(a, q, w, gi, gd, min(args.cpu_sample, nq),
                                                                  min(args.one_thread_sample, nq))
        assert entry == info["entry"], "entry node differs from the oracle's"
        log(f"oracle on CPU: {cpu['value']:,.0f} queries/s with {cpu['cores']} threads (nproc {cpu['nproc']}); "
            f"GPU answers oracle-exact on the sample: {exact}")
    R = info["R"]
    full_counts = ocounts["evaluations"] if ocounts is not None and ocounts["queries"] == nq else None
    traffic = measured_traffic(w.name, args.layout)
    kname = "search_resident<MetricU8>" if w.index.dtype == "u8" else "search_resident<MetricF32>"
    roofline = roofline_of(main_res, w, R, full_counts, traffic, kname)
    if full_counts is not None:
        roofline["expansions_match_oracle"] = ocounts["expansions"] == st["expansions"]
    if not args.no_gather_ceiling and args.layout == "vectors-first" and w.index.dtype == "u8":
        gc = gather_ceiling(w.index.n, info["records_per_page"], info["page_bytes"], 128)
        if gc is not None:
            roofline["gather_ceiling_gbs"] = gc["gbs"]
            roofline["frac_of_gather_ceiling"] = round(roofline["achieved"] / gc["gbs"], 4)
            log(f"random 128-B gather ceiling: {gc['gbs']:,.0f} GB/s; achieved {roofline['achieved']:,.0f} GB/s")
    recall = None
    if args.recall_sample > 0:
        recall = recall_at_k(a["x"], q, gi, w.k, min(args.recall_sample, nq))
        log(f"recall@{w.k} on {recall['queries']} queries: {recall['value']}")

    resident_legs = []
    # ------------------------------------------------------------ small index
    if not args.no_small and w.name != "u8-10k-hbm":
        ws = WORKLOADS["u8-10k-hbm"]
        a_s = index_arrays(ws.index)
        q_s = query_array(ws.index, ws.queries)
        r = resident_leg(torch, g, a_s, q_s, ws, "vectors-first", args.steps, args.warmup)
        cb, ex, _, oc, _, _ = cpu_baseline(a_s, q_s, ws, r["ids"], r["dists"], len(q_s), len(q_s))
        resident_legs.append({
            "workload": ws.name, "queries": len(q_s),
            "value": round(len(q_s) * args.steps / r["elapsed"], 1), "unit": "queries/s",
            "ms_per_step": round(r["elapsed"] * 1e3 / args.steps, 4), "steps": args.steps,
            "oracle_exact": ex, "roofline": roofline_of(r, ws, ws.index.R, oc["evaluations"], None,
                                                        "search_resident<MetricU8>"),
            "cpu_baseline": cb})
        log(f"{ws.name}: oracle-exact {ex}")

    # ------------------------------------------------------------------ paged
    paged = None
    miss_gbs = None
    if args.paged_sample != 0 and w.name == "u8-1m-hbm":
        link = host_link_peak_gbs(torch)
        legs = []
        placements = {}
        vfirst = args.layout == "vectors-first"

        def placement(nq_leg):
            k = cluster_count(args.paged_clusters, nq_leg)
            if k and k not in placements:
                t0 = time.perf_counter()
                placements[k] = g.cluster_order(a["x"], k)
                log(f"cluster placement ({k} clusters) in {time.perf_counter() - t0:.2f} s")
            return placements.get(k)

        def check(leg, pi, pd, pq, wl):
            # every paged answer must equal the resident kernel's on the same queries
            if wl.queries == w.queries:
                leg["equals_resident"] = bool(np.array_equal(pi, gi[:len(pq)]) and np.array_equal(pd, gd[:len(pq)]))
            if exact is not None and wl.queries == w.queries and len(pq) <= args.cpu_sample:
                leg["oracle_exact"] = bool(exact and leg.get("equals_resident"))
            log(f"paged {wl.name} ({len(pq)} queries) {leg['label']} {leg['placement']}: {leg['qps']:,.0f} q/s, "
                f"hit rate {leg['hit_rate']:.3f}, miss service {leg['miss_service_gbs']} GB/s")

        clustered = args.paged_clusters != 0
        w3 = WORKLOADS["u8-1m-cache10-lat0"]
        n3 = w3.queries.nq if args.paged_sample < 0 else min(args.paged_sample, w3.queries.nq)
        # C3 legs: split-phase and blocking in the same shape (one query per wave),
        # the identity placement, the default shape (as many queries as the pins
        # allow, 4 per wave), host-scheduled lanes (40), the GPU resume queue (40 lanes)
        plan = [(0, clustered, "split-phase", SHAPE_C3), (1, clustered, "blocking", SHAPE_C3),
                (0, False, "split-phase, identity placement", SHAPE_C3),
                (0, clustered, "split-phase, default shape", {}),
                (2, clustered, "host-scheduled", SHAPE_HOST),
                (3, clustered, "gpu resume queue", SHAPE_QUEUE)]
        for mode, use_cl, label, shape in plan:
            if use_cl is False and not clustered and label.endswith("identity placement"):
                continue
            if not fits(f"{w3.name} {label}", 6 + 3.0 * args.paged_repeats):
                continue
            cl = placement(n3) if use_cl else None
            leg, pi, pd, pq = paged_leg(torch, g, a, w3, n3, qps, mode, vfirst, args.paged_repeats, cl,
                                        label=label, **shape)
            check(leg, pi, pd, pq, w3)
            legs.append(leg)
        by_label = {l["label"]: l for l in legs}
        if by_label:
            miss_gbs = legs[0]["miss_service_gbs"]
        paged = {"host_link_peak_gbs": round(link, 1), "legs": legs}
        if "split-phase" in by_label and "blocking" in by_label:
            paged["split_phase_vs_blocking"] = round(by_label["split-phase"]["qps"] / by_label["blocking"]["qps"], 3)
        if "split-phase" in by_label and "split-phase, identity placement" in by_label:
            paged["clusters_vs_identity"] = round(
                by_label["split-phase"]["qps"] / by_label["split-phase, identity placement"]["qps"], 3)
        if "split-phase" in by_label and "split-phase, default shape" in by_label:
            paged["tuned_vs_default_shape"] = round(
                by_label["split-phase"]["qps"] / by_label["split-phase, default shape"]["qps"], 3)
        if "split-phase" in by_label and "host-scheduled" in by_label:
            paged["gpu_vs_host_scheduled"] = round(
                by_label["split-phase"]["qps"] / by_label["host-scheduled"]["qps"], 3)

        # equal-wave comparison: both modes get the split-phase default's query
        # waves; split-phase then holds oversub times more queries in flight
        if args.ablation_sample > 0:
            lats = [float(x) for x in args.ablation_latencies.split(",") if x.strip()]
            na = min(args.ablation_sample, w3.queries.nq)
            slots = int(w3.cache_frac * int(np.ceil(w3.index.n / w3.index.records_per_page)))
            waves = max(1, min(slots // (2 * 32), na) // w3.oversub)
            rows = []
            for lat in lats:
                row = {"latency_us": lat, "query_waves": waves,
                       "little_law_requests": round(link * 1e9 * lat * 1e-6 / 4096, 1)}
                for mode in (0, 1):
                    if not fits(f"equal-wave {MODES[mode]} at {lat} us", 4 + 2.5 * args.paged_repeats):
                        continue
                    cl = placement(na) if clustered else None
                    leg, pi, pd, pq = paged_leg(torch, g, a, w3, na, qps, mode, vfirst, args.paged_repeats, cl,
                                                warmup_nq=1000, query_waves=waves, latency_us=lat,
                                                label=f"equal waves, {MODES[mode]}")
                    check(leg, pi, pd, pq, w3)
                    row[MODES[mode]] = {k: leg[k] for k in ("qps", "qps_runs", "kernel_ms", "hit_rate",
                                                            "miss_service_gbs", "proxy_peak", "equals_resident")
                                        if k in leg}
                    row[MODES[mode]]["live_queries"] = waves * (w3.oversub if mode == 0 else 1)
                if "split-phase" in row and "blocking" in row:
                    row["split_phase_vs_blocking"] = round(row["split-phase"]["qps"] / row["blocking"]["qps"], 3)
                rows.append(row)
            paged["equal_wave_ablation"] = {
                "queries": na, "runs_per_point": args.paged_repeats,
                "blocking_outstanding_cap": waves * 32, "rows": rows}

        # C4: 100k queries, 20 us
        w4 = WORKLOADS["u8-1m-cache10-lat20"]
        n4 = w4.queries.nq if args.paged_sample < 0 else min(args.paged_sample, w4.queries.nq)
        if fits(w4.name, 8 + 15.0 * args.large_repeats * n4 / 100000):
            cl = placement(n4) if clustered else None
            leg, pi, pd, pq = paged_leg(torch, g, a, w4, n4, qps, 0, vfirst,
                                        args.large_repeats if n4 > 20000 else args.paged_repeats, cl,
                                        warmup_nq=10000, **SHAPE_C4)
            check(leg, pi, pd, pq, w4)
            if packed_main is not None:   # these queries differ from the resident batch: the oracle checks a slice
                ns = min(args.f32_cpu_sample, len(pq))
                oi, od4, _, _ = packed_main.search(pq[:ns], w4.k, w4.L, w4.W, info["entry"],
                                                   threads=oracle_threads()[0])
                leg["oracle_exact"] = bool(np.array_equal(pi[:ns], oi) and np.array_equal(pd[:ns], od4))
                leg["oracle_checked_queries"] = ns
            # what the host link allows at this hit rate, and what 2x of resident would need
            bpq = leg["pages_served"] * 4096 / max(1, leg["queries"])
            acc_pq = None
            leg["link_bound_qps"] = round(link * 1e9 / bpq, 1)
            if ocounts is not None and ocounts["queries"] > 0:
                acc_pq = (ocounts["expansions"] + ocounts["evaluations"]) / ocounts["queries"]
            if acc_pq:
                target = qps / 2
                allowed_misses = link * 1e9 / target / 4096
                leg["target_qps_2x_of_resident"] = round(target, 1)
                leg["record_accesses_per_query"] = round(acc_pq, 1)
                leg["hit_rate_needed_for_target"] = round(max(0.0, 1 - allowed_misses / acc_pq), 5)
            legs.append(leg)

    # --------------------------------------------------- 10M float32 index
    if args.f32_sample != 0:
        wr, wp = WORKLOADS["f32-10m-hbm"], WORKLOADS["f32-10m-cache5-lat20"]
        est_gen = 5 if index_cached(wr.index) else 90
        if fits(wr.name, est_gen + 40):
            log(f"{wr.name}: loading or generating the index")
            af = index_arrays(wr.index)
            qf = query_array(wr.index, wr.queries)
            if args.f32_sample > 0:
                qf = qf[:args.f32_sample]
            r = resident_leg(torch, g, af, qf, wr, "vectors-first", max(3, args.steps // 4), 1)
            rqps = len(qf) * max(3, args.steps // 4) / r["elapsed"]
            ftraffic = measured_traffic(wr.name, "vectors-first")
            fleg = {"workload": wr.name, "queries": len(qf),
                    "value": round(rqps, 1), "unit": "queries/s",
                    "ms_per_step": round(r["elapsed"] * 1e3 / max(3, args.steps // 4), 3),
                    "steps": max(3, args.steps // 4),
                    "roofline": roofline_of(r, wr, wr.index.R, None, ftraffic, "search_resident<MetricF32>"),
                    "counters": {k: r["stats"][k] for k in ("evaluations", "reevaluations", "expansions",
                                                            "iterations")}}
            if ftraffic:
                fleg["achieved_hbm_gbs"] = fleg["roofline"]["traffic_gbs"]
            packed = None
            if args.f32_cpu_sample > 0 and fits(f"{wr.name} oracle", 60):
                from oracle import load
                t0 = time.perf_counter()
                packed = load().pack(af["x"], af["graph"])
                log(f"{wr.name}: oracle pages packed in {time.perf_counter() - t0:.1f} s")
                ns = min(args.f32_cpu_sample, len(qf))
                cb, ex, entry, oc, (oids_f, od_f), _ = cpu_baseline(af, qf, wr, r["ids"], r["dists"], ns,
                                                                    ns // 10, packed=packed)
                fleg["cpu_baseline"] = cb
                fleg["oracle_exact"] = ex
                fleg["oracle_checked_queries"] = ns
                log(f"{wr.name}: {rqps:,.0f} q/s resident; oracle-exact on {ns}: {ex}")
            resident_legs.append(fleg)
            if not args.no_f32_paged and fits(wp.name, 30 + 52.0 * (args.large_repeats + 0.1) * len(qf) / 100000):
                t0 = time.perf_counter()
                fcl = g.cluster_order(af["x"], args.f32_clusters) if args.f32_clusters else None
                log(f"{wp.name}: cluster placement ({args.f32_clusters}) in {time.perf_counter() - t0:.2f} s")
                leg, pi, pd, _ = paged_leg(torch, g, af, wp, len(qf), rqps, 0, True,
                                           args.large_repeats if len(qf) > 20000 else args.paged_repeats,
                                           fcl, warmup_nq=10000, **SHAPE_C5)
                leg["equals_resident"] = bool(np.array_equal(pi, r["ids"]) and
                                              np.array_equal(pd.view(np.uint32), r["dists"].view(np.uint32)))
                if packed is not None:
                    ns = fleg["oracle_checked_queries"]
                    leg["oracle_exact"] = bool(np.array_equal(pi[:ns], oids_f) and
                                               np.array_equal(pd[:ns].view(np.uint32), od_f.view(np.uint32)))
                    leg["oracle_checked_queries"] = ns
                log(f"paged {wp.name}: {leg['qps']:,.0f} q/s, hit rate {leg['hit_rate']:.3f}, "
                    f"miss service {leg['miss_service_gbs']} GB/s (resident {rqps:,.0f} q/s)")
                if paged is None:
                    paged = {"host_link_peak_gbs": round(host_link_peak_gbs(torch), 1), "legs": []}
                paged["legs"].append(leg)
            del packed, af

    out = {
        "metric": METRIC, "value": round(qps, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.index.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "n": w.index.n, "D": w.index.D, "R": R, "nq": nq,
                   "k": w.k, "L": w.L, "W": w.W, "record_bytes": info["record_bytes"],
                   "records_per_page": info["records_per_page"], "page_layout": args.layout,
                   "cache_frac": w.cache_frac, "resident": bool(info["resident"])},
        "other_layout": other,
        "host_buffers": host_buffers,
        "oracle_exact": exact,
        "recall": recall,
        "achieved_hbm_gbs": roofline.get("traffic_gbs"),
        "achieved_hbm_frac": roofline.get("traffic_frac"),
        "algorithmic_gbs": roofline["achieved"],
        "miss_service_gbs": miss_gbs,
        "counters": {k: st[k] for k in ("evaluations", "reevaluations", "expansions", "iterations")},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "resident_legs": resident_legs,
        "paged": paged,
        "skipped": skipped,
        "paper_context": PAPER_CONTEXT,
        "bench_s": round(time.perf_counter() - T_START, 1),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
