"""The C ABI library loads, exports every declared symbol, and rejects bad
arguments before touching a device (runs without a GPU)."""
import ctypes
import re
from pathlib import Path

import numpy as np
import pytest

import paper_2607_04415_amd as g

HEADER = Path(__file__).resolve().parents[1] / "include" / "gorio.h"


@pytest.fixture(scope="module")
def lib():
    if not g.LIB_PATH.exists():
        from paper_2607_04415_amd import _build
        _build.build()
    return g.lib()


def declared_functions():
    text = HEADER.read_text()
    return sorted(set(re.findall(r"^\s*(?:gorio_status|void|const char \*)\s*(gorio_\w+)\s*\(",
                                 text, re.M)))


def test_header_declares_what_binding_expects():
    assert declared_functions() == sorted(g.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_library_loads_after_torchs_hip_runtime(lib):
    """torch brings its own HIP runtime, which a process loads first; the
    library may use only what that runtime exports (a symbol of a newer HIP
    release leaves the library unloadable there)."""
    import subprocess
    import sys
    code = ("import ctypes, torch; "
            f"ctypes.CDLL({str(g.LIB_PATH)!r}); print('loaded')")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "loaded" in r.stdout, r.stderr[-2000:]


def test_buffers_are_checked_before_the_library_sees_them():
    """Plain pointers cross the ABI, so the binding refuses a buffer of the
    wrong element type, one that is not contiguous, or one too small."""
    import torch
    chk = g._check_buffer
    chk("q", np.zeros((4, 8), np.uint8), 32, ("uint8",))
    chk("ids", torch.zeros((4, 3), dtype=torch.int32), 12, ("int32", "uint32"))
    with pytest.raises(ValueError, match="needs 33"):
        chk("q", np.zeros((4, 8), np.uint8), 33, ("uint8",))
    with pytest.raises(TypeError, match="float32"):
        chk("q", np.zeros((4, 8), np.float64), 32, ("float32",))
    with pytest.raises(ValueError, match="contiguous"):
        chk("q", np.zeros((8, 4), np.uint8).T, 32, ("uint8",))
    with pytest.raises(ValueError, match="contiguous"):
        chk("ids", torch.zeros((3, 4), dtype=torch.int32).t(), 12, ("int32",))
    with pytest.raises(ValueError, match="needs 13"):
        chk("ids", torch.zeros((4, 3), dtype=torch.int32), 13, ("int32",))
    with pytest.raises(ValueError, match="None"):
        chk("dists", None, 1, ("int32",))


def test_struct_sizes_match_header():
    # gorio_stats: 2 doubles + 11 uint64; gorio_page_layout: 4 uint32 + pointer
    assert ctypes.sizeof(g.Stats) == 2 * 8 + 11 * 8
    assert ctypes.sizeof(g.PageLayout) == 4 * 4 + 8


def _build(lib, dtype=0, n=10, D=8, R=4, layout=None, entry=g.NO_EDGE, vectors=True, graph=True):
    x = np.zeros((max(n, 1), max(D, 1)), np.uint8)
    gr = np.zeros((max(n, 1), max(R, 1)), np.uint32)
    h = ctypes.c_void_p()
    st = lib.gorio_build_index(dtype, x.ctypes.data if vectors else None, n, D,
                               gr.ctypes.data if graph else None, R,
                               ctypes.byref(layout) if layout is not None else None, entry,
                               ctypes.byref(h))
    return st, h


@pytest.mark.parametrize("kw", [
    dict(dtype=7), dict(n=0), dict(n=1 << 31), dict(R=0), dict(R=257), dict(D=0), dict(D=6),
    dict(D=516), dict(dtype=1, D=257), dict(entry=10), dict(vectors=False), dict(graph=False),
    dict(layout=g.PageLayout(4100, 0, 0, 0, None)),        # page size not a multiple of 16
    dict(layout=g.PageLayout(4096, 10, 0, 0, None)),       # record smaller than its contents
    dict(layout=g.PageLayout(4096, 26, 0, 0, None)),       # record not a multiple of 4
    dict(layout=g.PageLayout(4096, 0, 1000, 0, None)),     # too many records per page
    dict(layout=g.PageLayout(4096, 0, 0, 3, None)),        # unknown arrangement
    dict(D=4, R=4, layout=g.PageLayout(4096, 24, 0, 1, None)),  # vectors first: 16 + 4 + 16 > 24
])
def test_build_rejects_bad_arguments(lib, kw):
    st, h = _build(lib, **kw)
    assert st == g.EINVAL
    assert not h.value
    assert lib.gorio_last_error().decode()


def test_null_handles(lib):
    assert lib.gorio_set_cache(None, 0) == g.EINVAL
    assert lib.gorio_set_backing(None, 0.0, 0, 1, 0) == g.EINVAL
    assert lib.gorio_search(None, None, 0, 1, 1, 1, None, None, None, None) == g.EINVAL
    assert lib.gorio_index_info_get(None, None) == g.EINVAL
    assert lib.gorio_copy_pages(None, 0, 0, None) == g.EINVAL
    lib.gorio_free_index(None)


def test_build_needs_out_pointer(lib):
    x = np.zeros((4, 4), np.uint8)
    gr = np.zeros((4, 2), np.uint32)
    assert lib.gorio_build_index(0, x.ctypes.data, 4, 4, gr.ctypes.data, 2, None, g.NO_EDGE, None) == g.EINVAL


def test_cluster_order_rejects_bad_arguments(lib):
    """Argument checks come before any device work (no GPU needed)."""
    x = np.zeros((10, 4), np.uint8)
    n2s = np.empty(10, np.uint32)
    cent = np.empty((16, 4), np.float32)
    p = (x.ctypes.data, n2s.ctypes.data, cent.ctypes.data)
    for dt, n, D, K, it in ((0, 10, 4, 0, 2), (0, 10, 4, 11, 2), (0, 10, 4, 2, 65), (0, 0, 4, 1, 1),
                            (0, 10, 0, 2, 1), (0, 10, 1025, 2, 1), (5, 10, 4, 2, 1)):
        assert lib.gorio_cluster_order(dt, p[0], n, D, K, it, p[1], p[2]) == g.EINVAL
        assert lib.gorio_last_error().decode()
    assert lib.gorio_cluster_order(0, None, 10, 4, 2, 1, p[1], p[2]) == g.EINVAL
    assert lib.gorio_cluster_order(0, p[0], 10, 4, 2, 1, None, p[2]) == g.EINVAL
    assert lib.gorio_set_query_order(None, None, 0) == g.EINVAL
