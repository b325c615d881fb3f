"""Python binding of the gfx950 paged graph beam-search library (libgorio.so).

Argument marshalling only: every step of a search runs in the library's HIP
kernels.  The binding refuses to work when the library is not built.
Device arrays are torch tensors on a ROCm device; host arrays are numpy.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import numpy as np

_PKG = Path(__file__).resolve().parent
LIB_PATH = _PKG / "libgorio.so"

OK, EINVAL, ENOMEM, EDEVICE, ETIMEOUT, EUNSUPPORTED = range(6)
U8, F32 = 0, 1
LAYOUT_DEFAULT, LAYOUT_VECTORS_FIRST, LAYOUT_CONTIGUOUS = 0, 1, 2
NO_EDGE = 0xFFFFFFFF
_STATUS = {0: "OK", 1: "EINVAL", 2: "ENOMEM", 3: "EDEVICE", 4: "ETIMEOUT", 5: "EUNSUPPORTED"}


class GorioError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


class PageLayout(ctypes.Structure):
    _fields_ = [("page_bytes", ctypes.c_uint32), ("record_bytes", ctypes.c_uint32),
                ("records_per_page", ctypes.c_uint32), ("arrangement", ctypes.c_uint32),
                ("node_to_slot", ctypes.c_void_p)]


class Stats(ctypes.Structure):
    _fields_ = [("kernel_ms", ctypes.c_double), ("wall_ms", ctypes.c_double)] + [
        (f, ctypes.c_uint64) for f in ("evaluations", "reevaluations", "expansions", "iterations",
                                       "hits", "misses", "pages_served", "bytes_served",
                                       "parks", "resumes", "proxy_peak")]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


class IndexInfo(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("n", ctypes.c_uint64), ("D", ctypes.c_uint32),
                ("R", ctypes.c_uint32), ("page_bytes", ctypes.c_uint32),
                ("record_bytes", ctypes.c_uint32), ("records_per_page", ctypes.c_uint32),
                ("vectors_first", ctypes.c_int), ("num_pages", ctypes.c_uint64), ("index_bytes", ctypes.c_uint64),
                ("entry", ctypes.c_uint32), ("resident", ctypes.c_int),
                ("cache_slots", ctypes.c_uint64), ("device", ctypes.c_int)]

    def as_dict(self) -> dict:
        return {f: getattr(self, f) for f, _ in self._fields_}


# every symbol include/gorio.h declares
EXPORTS = ("gorio_build_index", "gorio_set_cache", "gorio_set_backing", "gorio_set_query_order",
           "gorio_search", "gorio_search_noalloc", "gorio_index_info_get", "gorio_copy_pages", "gorio_locality_order",
           "gorio_cluster_order", "gorio_set_scheduler", "gorio_free_index", "gorio_last_error")

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise RuntimeError(f"{LIB_PATH} is missing: build the HIP library first "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        L = ctypes.CDLL(str(LIB_PATH))
        v, u32, u64, i32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int
        L.gorio_build_index.restype = i32
        L.gorio_build_index.argtypes = [i32, v, u64, u32, v, u32, ctypes.POINTER(PageLayout), u32,
                                        ctypes.POINTER(v)]
        L.gorio_set_cache.restype = i32
        L.gorio_set_cache.argtypes = [v, u64]
        L.gorio_set_backing.restype = i32
        L.gorio_set_backing.argtypes = [v, ctypes.c_double, u32, u32, i32]
        L.gorio_set_scheduler.restype = i32
        L.gorio_set_scheduler.argtypes = [v, u32, u32]
        L.gorio_search.restype = i32
        L.gorio_search.argtypes = [v, v, u64, u32, u32, u32, v, v, ctypes.POINTER(Stats), v]
        L.gorio_search_noalloc.restype = i32
        L.gorio_search_noalloc.argtypes = [v, v, u64, u32, u32, u32, v, v, ctypes.POINTER(Stats), v]
        L.gorio_index_info_get.restype = i32
        L.gorio_index_info_get.argtypes = [v, ctypes.POINTER(IndexInfo)]
        L.gorio_copy_pages.restype = i32
        L.gorio_copy_pages.argtypes = [v, u64, u64, v]
        L.gorio_locality_order.restype = i32
        L.gorio_locality_order.argtypes = [v, u64, u32, u32, u32, v]
        L.gorio_cluster_order.restype = i32
        L.gorio_cluster_order.argtypes = [i32, v, u64, u32, u32, u32, v, v]
        L.gorio_set_query_order.restype = i32
        L.gorio_set_query_order.argtypes = [v, v, u32]
        L.gorio_free_index.restype = None
        L.gorio_free_index.argtypes = [v]
        L.gorio_last_error.restype = ctypes.c_char_p
        L.gorio_last_error.argtypes = []
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise GorioError(status, lib().gorio_last_error().decode())


def _ptr(a):
    """Data pointer of a numpy array or a torch tensor (None passes through)."""
    if a is None:
        return None
    if isinstance(a, np.ndarray):
        return a.ctypes.data
    return a.data_ptr()


def _check_buffer(name: str, a, count: int, dtypes: tuple):
    """The C ABI takes plain pointers and cannot check what they hold: a
    buffer of the wrong element type, not C-contiguous, or with fewer than
    `count` elements is refused here, before the library reads or writes it."""
    if a is None:
        raise ValueError(f"{name} is None")
    if isinstance(a, np.ndarray):
        dt, size, contiguous = a.dtype.name, a.size, a.flags.c_contiguous
    else:
        dt, size, contiguous = str(a.dtype).replace("torch.", ""), a.numel(), a.is_contiguous()
    if dt not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(dtypes)}, not {dt}")
    if not contiguous:
        raise ValueError(f"{name} must be C-contiguous")
    if size < count:
        raise ValueError(f"{name} holds {size} elements, the search needs {count}")


def locality_order(graph: np.ndarray, entry: int, records_per_page: int) -> np.ndarray:
    """node_to_slot placing graph neighbours in the same pages (gorio_locality_order)."""
    graph = np.ascontiguousarray(graph, dtype=np.uint32)
    out = np.empty(graph.shape[0], np.uint32)
    _check(lib().gorio_locality_order(graph.ctypes.data, graph.shape[0], graph.shape[1], int(entry),
                                      int(records_per_page), out.ctypes.data))
    return out


def cluster_order(vectors: np.ndarray, clusters: int, iterations: int = 4):
    """(node_to_slot, centroids): nodes placed cluster by cluster after
    `iterations` Lloyd steps of k-means on the GPU (gorio_cluster_order)."""
    vectors = np.ascontiguousarray(vectors)
    dt = U8 if vectors.dtype == np.uint8 else F32
    if dt == F32:
        vectors = np.ascontiguousarray(vectors, dtype=np.float32)
    n, D = vectors.shape
    n2s = np.empty(n, np.uint32)
    cent = np.empty((clusters, D), np.float32)
    _check(lib().gorio_cluster_order(dt, vectors.ctypes.data, n, D, int(clusters), int(iterations),
                                     n2s.ctypes.data, cent.ctypes.data))
    return n2s, cent


class Index:
    """A packed index (gorio_build_index) owned by the library."""

    def __init__(self, vectors: np.ndarray, graph: np.ndarray, page_bytes: int = 0,
                 record_bytes: int = 0, records_per_page: int = 0,
                 node_to_slot: np.ndarray | None = None, entry: int | None = None,
                 vectors_first: bool | None = None):
        """vectors_first: True = vectors-first pages, False = contiguous records,
        None = the library's default (vectors first)."""
        vectors = np.ascontiguousarray(vectors)
        graph = np.ascontiguousarray(graph, dtype=np.uint32)
        if vectors.dtype == np.uint8:
            self.dtype = U8
        elif vectors.dtype == np.float32:
            self.dtype = F32
        else:
            raise TypeError(f"vectors must be uint8 or float32, not {vectors.dtype}")
        n, D = vectors.shape
        if graph.shape[0] != n:
            raise ValueError("graph must have one row per vector")
        self._n2s = None if node_to_slot is None else np.ascontiguousarray(node_to_slot, np.uint32)
        arrangement = LAYOUT_DEFAULT if vectors_first is None else (
            LAYOUT_VECTORS_FIRST if vectors_first else LAYOUT_CONTIGUOUS)
        layout = PageLayout(page_bytes, record_bytes, records_per_page, arrangement, _ptr(self._n2s))
        h = ctypes.c_void_p()
        _check(lib().gorio_build_index(self.dtype, vectors.ctypes.data, n, D, graph.ctypes.data,
                                       graph.shape[1], ctypes.byref(layout),
                                       NO_EDGE if entry is None else entry, ctypes.byref(h)))
        self._h = h
        self.n, self.D, self.R = n, D, graph.shape[1]

    def close(self):
        if getattr(self, "_h", None):
            lib().gorio_free_index(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def info(self) -> dict:
        info = IndexInfo()
        _check(lib().gorio_index_info_get(self._h, ctypes.byref(info)))
        return info.as_dict()

    def set_cache(self, nbytes: int):
        _check(lib().gorio_set_cache(self._h, int(nbytes)))

    def set_backing(self, latency_us: float = 0.0, max_outstanding: int = 0, oversub: int = 1,
                    blocking: bool = False, mode: int | None = None):
        """mode: 0 split-phase, 1 blocking, 2 host-scheduled lanes, 3 GPU resume queue
        (default: from `blocking`)."""
        m = int(bool(blocking)) if mode is None else int(mode)
        _check(lib().gorio_set_backing(self._h, float(latency_us), int(max_outstanding),
                                       int(oversub), m))

    def set_scheduler(self, query_waves: int = 0, max_pending: int = 0):
        """Paged scheduler shape: most query waves and page requests per query (0 = default)."""
        _check(lib().gorio_set_scheduler(self._h, int(query_waves), int(max_pending)))

    def set_query_order(self, centroids: np.ndarray | None):
        """Paged searches admit queries by nearest centroid (None: index order)."""
        if centroids is None:
            _check(lib().gorio_set_query_order(self._h, None, 0))
            return
        c = np.ascontiguousarray(centroids, dtype=np.float32)
        _check(lib().gorio_set_query_order(self._h, c.ctypes.data, c.shape[0]))

    def pages(self, first: int = 0, count: int | None = None) -> np.ndarray:
        info = self.info
        count = info["num_pages"] - first if count is None else count
        out = np.empty(count * info["page_bytes"], np.uint8)
        _check(lib().gorio_copy_pages(self._h, first, count, out.ctypes.data))
        return out

    def search_into(self, queries, nq: int, k: int, L: int, W: int, ids, dists,
                    stream=None, stats: bool = True):
        """Raw call: queries/ids/dists are numpy arrays or device tensors
        (queries: nq x D of the index's element type; ids: nq x k int32 or
        uint32; dists: nq x k int32 for uint8 indexes, float32 for float32)."""
        if nq > 0:
            u8 = self.dtype == U8
            _check_buffer("queries", queries, nq * self.D, ("uint8",) if u8 else ("float32",))
            _check_buffer("ids", ids, nq * k, ("int32", "uint32"))
            _check_buffer("dists", dists, nq * k, ("int32",) if u8 else ("float32",))
        st = Stats()
        sp = None if stream is None else ctypes.c_void_p(stream)
        status = lib().gorio_search(self._h, _ptr(queries), nq, k, L, W, _ptr(ids), _ptr(dists),
                                    ctypes.byref(st) if stats else None, sp)
        if status != OK:
            err = GorioError(status, lib().gorio_last_error().decode())
            err.stats = st.as_dict() if stats else None   # counters up to the failure
            raise err
        return st.as_dict() if stats else None

    def search(self, queries, k: int, L: int, W: int, stream=None, stats: bool = True):
        """Search a batch.  numpy (or a CPU tensor) in -> numpy out; torch device
        tensor in -> tensors out."""
        if not isinstance(queries, np.ndarray) and not queries.is_cuda:
            queries = queries.numpy()
        if queries.shape[-1] != self.D or len(queries.shape) > 2:
            raise ValueError(f"queries must be (nq, {self.D}) or ({self.D},), not {tuple(queries.shape)}")
        if isinstance(queries, np.ndarray):
            queries = np.ascontiguousarray(queries)
            nq = queries.shape[0] if queries.ndim == 2 else 1
            ids = np.empty((nq, k), np.uint32)
            dists = np.empty((nq, k), np.int32 if self.dtype == U8 else np.float32)
        else:
            import torch
            queries = queries.contiguous()
            nq = queries.shape[0] if queries.dim() == 2 else 1
            ids = torch.empty((nq, k), dtype=torch.int32, device=queries.device)
            dists = torch.empty((nq, k), dtype=torch.int32 if self.dtype == U8 else torch.float32,
                                device=queries.device)
            if stream is None:
                stream = torch.cuda.current_stream(queries.device).cuda_stream
        st = self.search_into(queries, nq, k, L, W, ids, dists, stream=stream, stats=stats)
        return ids, dists, st
