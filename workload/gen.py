"""Seeded workload generator (inputs only).

Vectors: a Gaussian mixture drawn with numpy's PCG64 generator.
  * uint8: centres uniform in [40, 215]^D, point = rint(centre + sigma * N(0, I))
    clipped to [0, 255].
  * float32: centres ~ N(0, I) normalised to unit length, point =
    normalise(centre + sigma * N(0, I)) computed in float64, then cast.
  Cluster labels are uniform over [0, C).  Queries are fresh draws from the
  same mixture (same centres) with their own seed.

Graph: see edges.c (sampled-nearest + random edges, counter-based streams).

Arrays are cached on disk keyed by the full parameter set, so repeated calls in
one machine session cost a file read.
"""
from __future__ import annotations

import ctypes
import dataclasses
import hashlib
import json
import os
import sys
import subprocess
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
_EDGES_SRC = _HERE / "edges.c"
_EDGES_SO = _HERE / "_edges.so"
_CHUNK = 1 << 16


@dataclasses.dataclass(frozen=True)
class IndexSpec:
    n: int
    D: int
    dtype: str            # "u8" or "f32"
    clusters: int
    sigma: float
    r_near: int
    r_rand: int
    sample: int = 1024
    seed: int = 1

    @property
    def R(self) -> int:
        return self.r_near + self.r_rand

    @property
    def vec_bytes(self) -> int:
        return self.D * (1 if self.dtype == "u8" else 4)

    @property
    def record_bytes(self) -> int:
        # vector | u32 degree | R x u32 neighbour ids
        return self.vec_bytes + 4 + 4 * self.R

    @property
    def records_per_page(self) -> int:
        return 4096 // self.record_bytes

    @property
    def pages(self) -> int:
        rpp = self.records_per_page
        return (self.n + rpp - 1) // rpp


@dataclasses.dataclass(frozen=True)
class QuerySpec:
    nq: int
    seed: int


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: IndexSpec
    queries: QuerySpec
    k: int
    L: int
    W: int
    cache_frac: float = 1.0      # fraction of index pages the HBM cache holds
    latency_us: float = 0.0      # injected per-page-request latency of the backing store
    oversub: int = 1             # query slots per resident wave (paged mode)
    description: str = ""


_U8_10K = IndexSpec(n=10_000, D=128, dtype="u8", clusters=16, sigma=20.0,
                    r_near=16, r_rand=16, seed=1001)
_U8_1M = IndexSpec(n=1_000_000, D=128, dtype="u8", clusters=256, sigma=20.0,
                   r_near=32, r_rand=32, seed=1002)
_F32_10M = IndexSpec(n=10_000_000, D=96, dtype="f32", clusters=1024, sigma=0.05,
                     r_near=32, r_rand=32, seed=1005)

WORKLOADS = {
    w.name: w for w in [
        Workload("u8-10k-hbm", _U8_10K, QuerySpec(1_000, 2001), k=10, L=32, W=4,
                 description="10k x 128-d uint8, R=32, 1k queries, L=32 W=4, HBM-resident"),
        Workload("u8-1m-hbm", _U8_1M, QuerySpec(10_000, 2002), k=10, L=64, W=4,
                 description="1M x 128-d uint8, R=64, 10k queries, L=64 W=4, HBM-resident"),
        Workload("u8-1m-cache10-lat0", _U8_1M, QuerySpec(10_000, 2002), k=10, L=64, W=4,
                 cache_frac=0.10, latency_us=0.0, oversub=4,
                 description="1M uint8 index, 10% HBM page cache (cold), pinned-host "
                             "backing store, 0 us injected latency"),
        Workload("u8-1m-cache10-lat20", _U8_1M, QuerySpec(100_000, 2004), k=10, L=64, W=4,
                 cache_frac=0.10, latency_us=20.0, oversub=4,
                 description="1M uint8 index, 100k queries, 10% page cache, 20 us per "
                             "page request, 4x oversubscribed query slots"),
        Workload("f32-10m-hbm", _F32_10M, QuerySpec(100_000, 2005), k=10, L=128, W=8,
                 description="10M x 96-d float32, R=64, 100k queries, L=128 W=8, HBM-resident"),
        Workload("f32-10m-cache5-lat20", _F32_10M, QuerySpec(100_000, 2005), k=10, L=128, W=8,
                 cache_frac=0.05, latency_us=20.0, oversub=4,
                 description="10M x 96-d float32, R=64, 100k queries, L=128 W=8, 5% page "
                             "cache, 20 us per page request"),
    ]
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def cache_dir() -> Path:
    d = Path(os.environ.get("GORIO_WORKLOAD_CACHE", "/tmp/gorio_workloads"))
    d.mkdir(parents=True, exist_ok=True)
    return d


def _key(obj) -> str:
    blob = json.dumps(obj, sort_keys=True, default=str).encode()
    return hashlib.sha256(blob).hexdigest()[:20]


# --------------------------------------------------------------------------- #
# edge builder (C, OpenMP)
# --------------------------------------------------------------------------- #
def build_edges_lib(force: bool = False) -> Path:
    """Compile edges.c into _edges.so next to it."""
    if force or not _EDGES_SO.exists() or _EDGES_SO.stat().st_mtime < _EDGES_SRC.stat().st_mtime:
        tmp = _EDGES_SO.with_suffix(".so.tmp")
        subprocess.run(["gcc", "-O3", "-march=x86-64-v3", "-ffp-contract=off", "-fopenmp",
                        "-fPIC", "-shared", "-o", str(tmp), str(_EDGES_SRC)], check=True)
        os.replace(tmp, _EDGES_SO)
    return _EDGES_SO


_edges_lib = None


def _edges():
    global _edges_lib
    if _edges_lib is None:
        if not _EDGES_SO.exists():
            build_edges_lib()
        lib = ctypes.CDLL(str(_EDGES_SO))
        lib.gen_edges.restype = ctypes.c_int
        lib.gen_edges.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32,
                                  ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                  ctypes.c_uint64, ctypes.c_void_p]
        _edges_lib = lib
    return _edges_lib


def gen_graph(x: np.ndarray, labels: np.ndarray, clusters: int, sample: int,
              r_near: int, r_rand: int, seed: int) -> np.ndarray:
    n, D = x.shape
    x = np.ascontiguousarray(x)
    labels = np.ascontiguousarray(labels, dtype=np.uint32)
    members = np.argsort(labels, kind="stable").astype(np.uint32)
    counts = np.bincount(labels, minlength=clusters).astype(np.uint64)
    start = np.zeros(clusters + 1, np.uint64)
    np.cumsum(counts, out=start[1:])
    graph = np.empty((n, r_near + r_rand), np.uint32)
    dtype = 0 if x.dtype == np.uint8 else 1
    xs = np.ascontiguousarray(x[members])   # cluster by cluster: a node's samples are close in memory
    rc = _edges().gen_edges(dtype, xs.ctypes.data, n, D, start.ctypes.data, members.ctypes.data,
                            labels.ctypes.data, clusters, sample, r_near, r_rand, seed,
                            graph.ctypes.data)
    if rc != 0:
        raise RuntimeError(f"gen_edges failed with code {rc}")
    return graph


# --------------------------------------------------------------------------- #
# mixtures
# --------------------------------------------------------------------------- #
def _centres(rng: np.random.Generator, C: int, D: int, dtype: str) -> np.ndarray:
    if dtype == "u8":
        return rng.uniform(40.0, 215.0, size=(C, D))
    c = rng.standard_normal(size=(C, D))
    return c / np.linalg.norm(c, axis=1, keepdims=True)


def _progress(msg: str):
    """Progress of long generations on stderr (large workloads take minutes)."""
    print(f"[workload] {msg}", file=sys.stderr, flush=True)


def _draw(rng: np.random.Generator, centres: np.ndarray, count: int, sigma: float,
          dtype: str):
    C, D = centres.shape
    labels = rng.integers(0, C, size=count).astype(np.uint32)
    out = np.empty((count, D), np.uint8 if dtype == "u8" else np.float32)
    for s in range(0, count, _CHUNK):
        if count > 50 * _CHUNK and (s // _CHUNK) % 50 == 0:
            _progress(f"drawing vectors {s:,}/{count:,}")
        e = min(count, s + _CHUNK)
        v = centres[labels[s:e]] + sigma * rng.standard_normal(size=(e - s, D))
        if dtype == "u8":
            out[s:e] = np.clip(np.rint(v), 0, 255).astype(np.uint8)
        else:
            out[s:e] = (v / np.linalg.norm(v, axis=1, keepdims=True)).astype(np.float32)
    return labels, out


def _cached(tag: str, key_obj, make):
    d = cache_dir() / f"{tag}-{_key(key_obj)}"
    done = d / "DONE"
    if done.exists():
        names = done.read_text().split()
        return {k: np.load(d / f"{k}.npy", allow_pickle=False) for k in names}
    arrays = make()
    d.mkdir(parents=True, exist_ok=True)
    big = sum(v.nbytes for v in arrays.values()) > (1 << 30)
    for k, v in arrays.items():
        if big:
            _progress(f"saving {k} ({v.nbytes / 1e9:.2f} GB) to {d}")
        tmp = d / f"{k}.{os.getpid()}.tmp.npy"
        np.save(tmp, v)
        os.replace(tmp, d / f"{k}.npy")
    done.write_text(" ".join(arrays))
    return arrays


def _index_key(spec: IndexSpec) -> dict:
    # the edge builder's source is part of the key: a change to it never
    # reuses graphs it built before
    return {**dataclasses.asdict(spec), "edges_src": hashlib.sha256(_EDGES_SRC.read_bytes()).hexdigest()[:16]}


def index_cached(spec: IndexSpec) -> bool:
    """Whether index_arrays(spec) would load from the cache instead of generating."""
    return (cache_dir() / f"index-{_key(_index_key(spec))}" / "DONE").exists()


def index_arrays(spec: IndexSpec, use_cache: bool = True) -> dict:
    """{'x': n x D vectors, 'graph': n x R uint32, 'labels': n uint32, 'centres': C x D}."""
    def make():
        rng = np.random.default_rng(spec.seed)
        centres = _centres(rng, spec.clusters, spec.D, spec.dtype)
        labels, x = _draw(rng, centres, spec.n, spec.sigma, spec.dtype)
        if spec.n >= 1_000_000:
            _progress(f"building edges for {spec.n:,} nodes")
        graph = gen_graph(x, labels, spec.clusters, spec.sample, spec.r_near, spec.r_rand,
                          spec.seed)
        return {"x": x, "graph": graph, "labels": labels, "centres": centres}
    if not use_cache:
        return make()
    return _cached("index", _index_key(spec), make)


def query_array(spec: IndexSpec, q: QuerySpec) -> np.ndarray:
    """Queries from the same mixture as `spec` (same centres), own seed."""
    def make():
        rng = np.random.default_rng(spec.seed)
        centres = _centres(rng, spec.clusters, spec.D, spec.dtype)
        qrng = np.random.default_rng(q.seed)
        _, xq = _draw(qrng, centres, q.nq, spec.sigma, spec.dtype)
        return {"q": xq}
    return _cached("queries", [dataclasses.asdict(spec), dataclasses.asdict(q)], make)["q"]
