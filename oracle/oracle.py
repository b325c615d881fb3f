"""ctypes binding of the C oracle (gorio_oracle.c) -- TEST INFRASTRUCTURE ONLY.

Build: gcc -O2 -ffp-contract=off (no fused multiply-add, so float32 distances
follow the plain sequential recipe), no -ffast-math (keeps subnormals).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
SRC_PATH = _HERE / "gorio_oracle.c"
LIB_PATH = _HERE / "liboracle.so"

U8, F32 = 0, 1
NO_EDGE = 0xFFFFFFFF
ERRORS = {0: "ok", 1: "invalid argument", 2: "out of memory", 3: "invariant violated"}


def build(src: Path = SRC_PATH, out: Path = LIB_PATH) -> Path:
    """Compile the oracle into a shared library."""
    out = Path(out)
    tmp = out.with_name(out.name + f".{os.getpid()}.tmp")
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                    "-fPIC", "-shared", "-o", str(tmp), str(src)], check=True)
    os.replace(tmp, out)
    return out


class _Index(ctypes.Structure):
    _fields_ = [("pages", ctypes.c_void_p), ("n", ctypes.c_uint64), ("D", ctypes.c_uint32),
                ("R", ctypes.c_uint32), ("dtype", ctypes.c_int32),
                ("page_bytes", ctypes.c_uint32), ("record_bytes", ctypes.c_uint32),
                ("records_per_page", ctypes.c_uint32), ("node_to_slot", ctypes.c_void_p),
                ("entry", ctypes.c_uint32), ("vectors_first", ctypes.c_int32)]


class _Counts(ctypes.Structure):
    _fields_ = [("evaluations", ctypes.c_uint64), ("expansions", ctypes.c_uint64),
                ("iterations", ctypes.c_uint64)]


COUNTS_DTYPE = np.dtype([("evaluations", np.uint64), ("expansions", np.uint64),
                         ("iterations", np.uint64)])


def _ptr(a):
    return None if a is None else a.ctypes.data


class Oracle:
    """One loaded copy of the oracle library (tests may load mutated builds)."""

    def __init__(self, path: Path = LIB_PATH):
        lib = ctypes.CDLL(str(path))
        v, u32, u64, i32 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int32
        lib.orc_record_bytes.restype = u32
        lib.orc_record_bytes.argtypes = [i32, u32, u32, i32]
        lib.orc_num_pages.restype = u64
        lib.orc_num_pages.argtypes = [u64, u32]
        lib.orc_dist_u8.restype = u32
        lib.orc_dist_u8.argtypes = [v, v, u32]
        lib.orc_dist_f32.restype = ctypes.c_float
        lib.orc_dist_f32.argtypes = [v, v, u32]
        lib.orc_pack.restype = ctypes.c_int
        lib.orc_pack.argtypes = [i32, v, u64, u32, v, u32, u32, u32, u32, v, i32, v]
        lib.orc_medoid.restype = u32
        lib.orc_medoid.argtypes = [i32, v, u64, u32]
        lib.orc_search.restype = ctypes.c_int
        lib.orc_search.argtypes = [ctypes.POINTER(_Index), v, u64, u64, u32, u32, u32,
                                   v, v, v, v, u64, ctypes.c_int]
        self.lib = lib
        self.path = Path(path)

    # -- helpers ----------------------------------------------------------- #
    @staticmethod
    def dtype_code(x: np.ndarray) -> int:
        if x.dtype == np.uint8:
            return U8
        if x.dtype == np.float32:
            return F32
        raise TypeError(f"unsupported vector dtype {x.dtype}")

    def record_bytes(self, dtype: int, D: int, R: int, vectors_first: bool = False) -> int:
        return int(self.lib.orc_record_bytes(dtype, D, R, int(bool(vectors_first))))

    def dist(self, a: np.ndarray, b: np.ndarray):
        a = np.ascontiguousarray(a)
        b = np.ascontiguousarray(b, dtype=a.dtype)
        if a.dtype == np.uint8:
            return int(self.lib.orc_dist_u8(a.ctypes.data, b.ctypes.data, a.size))
        return np.float32(self.lib.orc_dist_f32(a.ctypes.data, b.ctypes.data, a.size))

    def medoid(self, x: np.ndarray) -> int:
        x = np.ascontiguousarray(x)
        return int(self.lib.orc_medoid(self.dtype_code(x), x.ctypes.data, x.shape[0], x.shape[1]))

    def pack(self, x: np.ndarray, graph: np.ndarray, page_bytes: int = 4096,
             record_bytes: int | None = None, records_per_page: int | None = None,
             node_to_slot: np.ndarray | None = None, vectors_first: bool = False) -> "PackedIndex":
        x = np.ascontiguousarray(x)
        graph = np.ascontiguousarray(graph, dtype=np.uint32)
        n, D = x.shape
        R = graph.shape[1]
        dt = self.dtype_code(x)
        vf = int(bool(vectors_first))
        rb = record_bytes or self.record_bytes(dt, D, R, vf)
        rpp = records_per_page or page_bytes // rb
        if node_to_slot is not None:
            node_to_slot = np.ascontiguousarray(node_to_slot, dtype=np.uint32)
        npages = int(self.lib.orc_num_pages(n, max(rpp, 1)))
        pages = np.zeros(npages * page_bytes, np.uint8)
        rc = self.lib.orc_pack(dt, x.ctypes.data, n, D, graph.ctypes.data, R, page_bytes, rb,
                               rpp, _ptr(node_to_slot), vf, pages.ctypes.data)
        if rc != 0:
            raise ValueError(f"orc_pack: {ERRORS.get(rc, rc)}")
        return PackedIndex(self, pages, n, D, R, dt, page_bytes, rb, rpp, node_to_slot, vf)


class PackedIndex:
    def __init__(self, orc: Oracle, pages, n, D, R, dtype, page_bytes, record_bytes, rpp,
                 node_to_slot, vectors_first=0):
        self.orc, self.pages, self.n, self.D, self.R = orc, pages, n, D, R
        self.dtype, self.page_bytes, self.record_bytes, self.rpp = dtype, page_bytes, record_bytes, rpp
        self.node_to_slot = node_to_slot
        self.vectors_first = vectors_first

    def _struct(self, entry: int) -> _Index:
        return _Index(self.pages.ctypes.data, self.n, self.D, self.R, self.dtype, self.page_bytes,
                      self.record_bytes, self.rpp, _ptr(self.node_to_slot), entry, self.vectors_first)

    def search(self, queries: np.ndarray, k: int, L: int, W: int, entry: int,
               threads: int = 1, debug: bool = False, trace_cap: int = 0):
        """Returns (ids [nq,k] uint32, dists [nq,k] int32|float32, counts [nq], trace|None)."""
        queries = np.ascontiguousarray(queries)
        if queries.ndim == 1:
            queries = queries[None, :]
        nq = queries.shape[0]
        ids = np.empty((nq, k), np.uint32)
        dists = np.empty((nq, k), np.int32 if self.dtype == U8 else np.float32)
        counts = np.zeros(nq, COUNTS_DTYPE)
        trace = np.full((nq, trace_cap), NO_EDGE, np.uint32) if trace_cap else None
        ix = self._struct(entry)

        def run(lo, hi):
            return self.orc.lib.orc_search(ctypes.byref(ix), queries.ctypes.data, lo, hi, k, L, W,
                                           ids.ctypes.data, dists.ctypes.data, counts.ctypes.data,
                                           _ptr(trace), trace_cap, int(debug))

        if threads <= 1 or nq < 2:
            rcs = [run(0, nq)]
        else:
            bounds = np.linspace(0, nq, threads + 1).astype(np.int64)
            with ThreadPoolExecutor(threads) as ex:
                rcs = list(ex.map(lambda t: run(int(bounds[t]), int(bounds[t + 1])), range(threads)))
        for rc in rcs:
            if rc != 0:
                raise RuntimeError(f"orc_search: {ERRORS.get(rc, rc)}")
        return ids, dists, counts, trace


_default = None


def load() -> Oracle:
    """The oracle built from this directory's source (builds it if missing)."""
    global _default
    if _default is None:
        if not LIB_PATH.exists() or LIB_PATH.stat().st_mtime < SRC_PATH.stat().st_mtime:
            build()
        _default = Oracle(LIB_PATH)
    return _default
