"""Benchmark: batched paged graph beam search on one MI355X.

One step = one gorio_search over the whole query batch of the workload (all
steps of the search path).  Default workload: 1,000,000 x 128-d uint8 vectors,
R = 64, 388-B records, 10 per 4 KB page, 10,000 queries, k = 10, L = 64, W = 4,
every page resident in HBM.

Prints one JSON line.  `value` is queries per second over the timed steps
(inputs already resident in HBM).  `roofline` prices the search kernel's
algorithmic bytes (expansions x (4 + 4R) + first-time evaluations x vector
bytes) against its average duration, measured with HIP events on the launch
stream.  `cpu_baseline` times the CPU oracle on a bounded sample.
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


def log(msg):
    print(msg, file=sys.stderr, flush=True)


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


def cpu_baseline(a, q, w, gpu_ids, gpu_dists, sample_nq: int, threads: int):
    """Time the CPU oracle on the first `sample_nq` queries with `threads` threads
    on disjoint shards; also check the GPU answers on that sample."""
    from oracle import load
    orc = load()
    packed = orc.pack(a["x"], a["graph"])
    entry = orc.medoid(a["x"])
    qs = q[:sample_nq]
    t0 = time.perf_counter()
    oids, od, oc, _ = packed.search(qs, w.k, w.L, w.W, entry, threads=threads)
    dt = time.perf_counter() - t0
    exact = bool(np.array_equal(oids, gpu_ids[:sample_nq]) and np.array_equal(od, gpu_dists[:sample_nq]))
    counts = {"queries": len(qs), "evaluations": int(oc["evaluations"].sum()),
              "expansions": int(oc["expansions"].sum())}
    return {
        "value": round(sample_nq / dt, 1), "unit": "queries/s", "cores": threads, "kind": "oracle",
        "sample": f"first {sample_nq} of {len(q)} queries of the same workload, "
                  f"{threads} threads on disjoint query shards, {dt:.2f} s wall",
    }, exact, entry, counts


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
        log(f"[bench] gather ceiling probe failed: {r.stderr.strip()}")
        return None
    d = json.loads(r.stdout.strip().splitlines()[-1])
    best = max(d[k]["gbs"] for k in d if k.startswith("rounds_"))
    return {"gbs": best, "vectors": d["vectors"], "waves": d["waves"],
            "depths_gbs": {k: d[k]["gbs"] for k in d if k.startswith("rounds_")}}


def cluster_count(arg: int, nq: int) -> int:
    """k-means clusters for a paged leg: `arg` if positive, none if 0, else by
    the leg's query count.  Queries are admitted cluster by cluster, so a
    larger batch can use smaller clusters before too few of its queries share
    each one (1M uint8 index, 10% cache: 256 clusters best at 10k queries,
    512 at 100k)."""
    if arg >= 0:
        return arg
    return 256 if nq <= 20000 else 512


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


def paged_leg(torch, g, a, w, nq_sample: int, resident_qps: float, blocking: bool = False,
              vectors_first: bool = False, repeats: int = 5, clusters=None):
    """Cold-cache paged searches over the first nq_sample queries of workload w:
    `repeats` timed runs, each after set_cache has emptied the cache; the
    figures are the median run's.  clusters = (node_to_slot, centroids): pages
    placed cluster by cluster and queries admitted cluster by cluster."""
    from workload import query_array
    q = query_array(w.index, w.queries)[:nq_sample]
    ix = g.Index(a["x"], a["graph"], vectors_first=vectors_first,
                 node_to_slot=None if clusters is None else clusters[0])
    if clusters is not None:
        ix.set_query_order(clusters[1])
    qd = torch.from_numpy(q).cuda()
    ids = torch.empty((len(q), w.k), dtype=torch.int32, device="cuda")
    dists = torch.empty((len(q), w.k), dtype=torch.int32 if q.dtype == np.uint8 else torch.float32,
                        device="cuda")
    runs = []
    for _ in range(max(1, repeats)):
        ix.set_cache(int(w.cache_frac * ix.info["index_bytes"]))      # empty cache
        ix.set_backing(latency_us=w.latency_us, oversub=1 if blocking else w.oversub, blocking=blocking)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st = ix.search_into(qd, len(q), w.k, w.L, w.W, ids, dists,
                            stream=torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        runs.append((time.perf_counter() - t0, st))
    runs.sort(key=lambda r: r[0])
    wall, st = runs[len(runs) // 2]
    ms = st["kernel_ms"]
    acc = st["hits"] + st["misses"]
    out = {"workload": w.name, "queries": len(q), "blocking": blocking,
           "placement": "identity" if clusters is None else f"clusters ({len(clusters[1])}, queries by cluster)",
           "cache_slots": ix.info["cache_slots"], "latency_us": w.latency_us,
           "oversub": 1 if blocking else w.oversub, "runs": len(runs),
           "qps": round(len(q) / wall, 1), "qps_runs": [round(len(q) / r[0], 1) for r in runs],
           "kernel_ms": round(ms, 2),
           "hit_rate": round(st["hits"] / max(1, acc), 4),
           "pages_served": st["pages_served"],
           "miss_service_gbs": round(st["bytes_served"] / (ms * 1e-3) / 1e9, 2),
           "parks": st["parks"], "resumes": st["resumes"],
           "vs_resident_qps": round(len(q) / wall / resident_qps, 5) if resident_qps else None}
    ix.close()
    return out, ids.cpu().numpy().view(np.uint32), dists.cpu().numpy(), q


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="u8-1m-hbm")
    ap.add_argument("--layout", choices=LAYOUTS, default="vectors-first",
                    help="page layout of the timed index (the other one is timed too and reported)")
    ap.add_argument("--no-other-layout", action="store_true",
                    help="do not time the other page layout")
    ap.add_argument("--cpu-sample", type=int, default=10000)
    ap.add_argument("--recall-sample", type=int, default=100,
                    help="queries whose recall@k against exact top-k is reported (0 = skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gather-ceiling", action="store_true",
                    help="skip the random-gather ceiling probe (microbench/gather_ceiling)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (counter calibration)")
    ap.add_argument("--paged-sample", type=int, default=-1,
                    help="queries of each paged configuration to run (-1 = its full query count, "
                         "0 = skip the paged legs)")
    ap.add_argument("--paged-clusters", type=int, default=-1,
                    help="paged legs: k-means clusters for page placement and query admission (0 = off, "
                         "-1 = by the leg's query count: 256 up to 20k queries, 512 above)")
    ap.add_argument("--paged-repeats", type=int, default=3,
                    help="cold-cache runs per paged leg of up to 20k queries (the median is reported); "
                         "larger legs run once")
    ap.add_argument("--f32-sample", type=int, default=0,
                    help="queries of the 10M x 96-d float32 paged configuration to run (0 = skip; "
                         "generating that index takes minutes the first time)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only (asked for {args.gpus}); "
              "the search shards by query across GPUs but no multi-GPU path is built.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_04415_amd as g
    from workload import WORKLOADS, index_arrays, query_array

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
    w = WORKLOADS[args.workload]
    log(f"[bench] workload {w.name}: {w.description}")
    t0 = time.perf_counter()
    a = index_arrays(w.index)
    q = query_array(w.index, w.queries)
    log(f"[bench] inputs ready in {time.perf_counter() - t0:.1f} s")
    qd = torch.from_numpy(q).cuda()
    nq = len(q)

    def timed(layout: str):
        """Build the index in `layout`, run the warm-up and the timed steps."""
        ix = g.Index(a["x"], a["graph"], vectors_first=layout == "vectors-first")
        info = ix.info
        if w.cache_frac < 1.0:
            ix.set_cache(int(w.cache_frac * info["index_bytes"]))
            ix.set_backing(latency_us=w.latency_us, oversub=w.oversub)
        ids = torch.empty((nq, w.k), dtype=torch.int32, device="cuda")
        dists = torch.empty((nq, w.k), dtype=torch.int32, device="cuda")
        stream = torch.cuda.current_stream().cuda_stream
        for _ in range(args.warmup):
            ix.search_into(qd, nq, w.k, w.L, w.W, ids, dists, stream=stream)
        # Timed steps are issued back to back on the stream, as a serving loop
        # would: no host round trip per batch (the call returns once the search
        # is queued).  HIP events recorded on the same stream around each call
        # give every launch's duration; the counters come from one more call
        # after the timed region.
        cur = torch.cuda.current_stream()
        events = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(cur)
            ix.search_into(qd, nq, w.k, w.L, w.W, ids, dists, stream=stream, stats=False)
            e1.record(cur)
            events.append((e0, e1))
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        kernel_ms = [a.elapsed_time(b) for a, b in events]
        stats = [ix.search_into(qd, nq, w.k, w.L, w.W, ids, dists, stream=stream)]
        ix.close()
        log(f"[bench] {layout}: {args.steps} steps: {elapsed * 1e3 / args.steps:.3f} ms/step, "
            f"{nq * args.steps / elapsed:,.0f} queries/s")
        return info, elapsed, kernel_ms, stats, ids, dists

    info, elapsed, kernel_ms, stats, ids, dists = timed(args.layout)
    ms_per_step = elapsed * 1e3 / args.steps
    qps = nq * args.steps / elapsed
    other = None
    if not args.no_other_layout:
        o_layout = [x for x in LAYOUTS if x != args.layout][0]
        _, o_el, o_kms, _, o_ids, o_d = timed(o_layout)
        other = {"layout": o_layout, "value": round(nq * args.steps / o_el, 1),
                 "ms_per_step": round(o_el * 1e3 / args.steps, 4),
                 "kernel_ms_avg": round(float(np.mean(o_kms)), 4),
                 "same_answers": bool(torch.equal(o_ids, ids) and torch.equal(o_d, dists))}

    gi = ids.cpu().numpy().view(np.uint32)
    gd = dists.cpu().numpy()
    cpu = None
    exact = None
    ocounts = None
    if not args.no_cpu_baseline:
        threads = min(os.cpu_count() or 1, 16)
        cpu, exact, entry, ocounts = cpu_baseline(a, q, w, gi, gd, min(args.cpu_sample, nq), threads)
        assert entry == info["entry"], "entry node differs from the oracle's"
        log(f"[bench] oracle on CPU: {cpu['value']:,.0f} queries/s with {threads} threads; "
            f"GPU answers oracle-exact on the sample: {exact}")

    # Algorithmic bytes: every expansion reads 4 + 4R bytes, every node of V
    # (first-time evaluations) its vector.  |V| is exact from the oracle's
    # counts when it ran on the whole batch; otherwise the GPU's evaluations
    # minus those it could not record in its visited filter (a lower bound:
    # an unrecorded evaluation may still be the node's first).
    st = stats[-1]
    R = info["R"]
    vec_bytes = w.index.vec_bytes
    if ocounts is not None and ocounts["queries"] == nq:
        first_evals, counts_source = ocounts["evaluations"], "oracle"
    else:
        first_evals, counts_source = st["evaluations"] - st["reevaluations"], "gpu lower bound"
    alg_bytes = st["expansions"] * (4 + 4 * R) + first_evals * vec_bytes
    avg_kernel_ms = float(np.mean(kernel_ms))
    achieved = alg_bytes / (avg_kernel_ms * 1e-3) / 1e9
    traffic = measured_traffic(w.name, args.layout)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic,
                "kernel": "search_resident<MetricU8>", "kernel_ms_avg": round(avg_kernel_ms, 4),
                "algorithmic_bytes_per_launch": int(alg_bytes),
                "algorithmic_counts": counts_source,
                "expansions_match_oracle": (None if counts_source != "oracle"
                                            else ocounts["expansions"] == st["expansions"])}

    if not args.no_gather_ceiling and args.layout == "vectors-first" and w.index.dtype == "u8":
        gc = gather_ceiling(w.index.n, info["records_per_page"], info["page_bytes"], 128)
        if gc is not None:
            roofline["gather_ceiling_gbs"] = gc["gbs"]
            roofline["frac_of_gather_ceiling"] = round(achieved / gc["gbs"], 4)
            log(f"[bench] random 128-B gather ceiling: {gc['gbs']:,.0f} GB/s "
                f"({gc['vectors']:,} vectors, {gc['waves']} waves); achieved {achieved:,.0f} GB/s")

    recall = None
    if args.recall_sample > 0:
        recall = recall_at_k(a["x"], q, gi, w.k, min(args.recall_sample, nq))
        log(f"[bench] recall@{w.k} on {recall['queries']} queries: {recall['value']}")

    paged = None
    miss_gbs = None
    if args.paged_sample != 0 and w.name == "u8-1m-hbm":
        link = host_link_peak_gbs(torch)
        legs = []
        placements = {}

        def placement(nq_leg):
            k = cluster_count(args.paged_clusters, nq_leg)
            if k and k not in placements:
                t0 = time.perf_counter()
                placements[k] = g.cluster_order(a["x"], k)
                log(f"[bench] cluster placement ({k} clusters) in {time.perf_counter() - t0:.1f} s")
            return placements.get(k)

        # C3 (10k queries, 0 us): split-phase and blocking; the identity
        # placement beside them; C4 (100k queries, 20 us): split-phase, one run
        clustered = args.paged_clusters != 0
        plan = [("u8-1m-cache10-lat0", False, clustered), ("u8-1m-cache10-lat0", True, clustered)]
        if clustered:
            plan.append(("u8-1m-cache10-lat0", False, False))   # identity placement, index order
        plan.append(("u8-1m-cache10-lat20", False, clustered))
        for name, blocking, use_clusters in plan:
            wl = WORKLOADS[name]
            nq_leg = wl.queries.nq if args.paged_sample < 0 else min(args.paged_sample, wl.queries.nq)
            cl = placement(nq_leg) if use_clusters else None
            reps = args.paged_repeats if nq_leg <= 20000 else 1
            leg, pi, pd, pq = paged_leg(torch, g, a, wl, nq_leg, qps, blocking,
                                        vectors_first=args.layout == "vectors-first",
                                        repeats=reps, clusters=cl)
            # the paged results must equal the resident results on the same queries
            if wl.queries == w.queries:
                leg["equals_resident"] = bool(np.array_equal(pi, gi[:len(pq)]) and np.array_equal(pd, gd[:len(pq)]))
            log(f"[bench] paged {name} ({len(pq)} queries) blocking={blocking} {leg['placement']}: "
                f"{leg['qps']:,.0f} q/s, hit rate {leg['hit_rate']:.3f}, miss service {leg['miss_service_gbs']} GB/s")
            legs.append(leg)
        miss_gbs = legs[0]["miss_service_gbs"]
        paged = {"host_link_peak_gbs": round(link, 1), "legs": legs,
                 "split_phase_vs_blocking": round(legs[0]["qps"] / max(1e-9, legs[1]["qps"]), 3)}
        if clustered:
            paged["clusters_vs_identity"] = round(legs[0]["qps"] / max(1e-9, legs[2]["qps"]), 3)

    if args.f32_sample > 0:
        wf = WORKLOADS["f32-10m-cache5-lat20"]
        log(f"[bench] {wf.name}: loading or generating the index")
        af = index_arrays(wf.index)
        qf = query_array(wf.index, wf.queries)[:args.f32_sample]
        # the same queries on the HBM-resident index: the reference answers and rate
        ixr = g.Index(af["x"], af["graph"], vectors_first=args.layout == "vectors-first")
        ri, rd, rst = ixr.search(torch.from_numpy(qf).cuda(), wf.k, wf.L, wf.W)
        torch.cuda.synchronize()
        ri, rd = ri.cpu().numpy().view(np.uint32), rd.cpu().numpy()
        rqps = len(qf) / (rst["kernel_ms"] * 1e-3)
        ixr.close()
        fclusters = None
        fk = cluster_count(args.paged_clusters, len(qf))
        if fk:
            t0 = time.perf_counter()
            fclusters = g.cluster_order(af["x"], fk)
            log(f"[bench] {wf.name}: cluster placement ({fk} clusters) in "
                f"{time.perf_counter() - t0:.1f} s")
        leg, pi, pd, _ = paged_leg(torch, g, af, wf, args.f32_sample, rqps,
                                   vectors_first=args.layout == "vectors-first", repeats=1, clusters=fclusters)
        leg["resident_kernel_qps"] = round(rqps, 1)
        leg["equals_resident"] = bool(np.array_equal(pi, ri) and np.array_equal(pd.view(np.uint32), rd.view(np.uint32)))
        log(f"[bench] paged {wf.name}: {leg['qps']:,.0f} q/s, hit rate {leg['hit_rate']:.3f}, "
            f"miss service {leg['miss_service_gbs']} GB/s (resident {rqps:,.0f} q/s)")
        if paged is None:
            paged = {"host_link_peak_gbs": round(host_link_peak_gbs(torch), 1), "legs": []}
        paged["legs"].append(leg)
        del af

    out = {
        "metric": METRIC, "value": round(qps, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": w.name, "n": w.index.n, "D": w.index.D, "R": R, "nq": nq,
                   "k": w.k, "L": w.L, "W": w.W, "record_bytes": info["record_bytes"],
                   "records_per_page": info["records_per_page"], "page_layout": args.layout,
                   "cache_frac": w.cache_frac, "resident": bool(info["resident"])},
        "other_layout": other,
        "oracle_exact": exact,
        "recall": recall,
        "achieved_hbm_gbs": roofline["achieved"],
        "miss_service_gbs": miss_gbs,
        "counters": {k: st[k] for k in ("evaluations", "reevaluations", "expansions", "iterations")},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "paged": paged,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
