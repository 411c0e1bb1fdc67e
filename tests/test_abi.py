"""The C ABI library loads and exports every symbol include/wl.h declares;
host-only argument checks (no GPU work is started by these calls)."""
import ctypes
import os
import re

import pytest

import paper_2607_02603_amd as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _ensure_built():
    if not os.path.exists(wl.LIB_PATH):
        from paper_2607_02603_amd import build
        build.build_wl()


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "wl.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wl_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for name in ("wl_refine_round", "wl_stable_coloring", "wl_stable_coloring_batched",
                 "wl_workspace_size", "wl_verify_stable", "wl_last_error"):
        assert name in syms


def test_library_exports_every_declared_symbol():
    _ensure_built()
    L = ctypes.CDLL(wl.LIB_PATH)
    for name in declared_symbols():
        assert hasattr(L, name), name
    assert sorted(wl.EXPORTED) == declared_symbols()


def _csr(n, nnz, rp32=True):
    s = wl.WlCsr()
    s.n = n
    s.nnz = nnz
    s.row_ptr32 = 8 if rp32 else None
    s.row_ptr64 = None if rp32 else 8
    s.col_idx = 16 if nnz else None
    s.weight = None
    return s


def test_workspace_size_host_only():
    _ensure_built()
    L = wl.lib()
    out = ctypes.c_uint64(0)
    s = _csr(1000, 5000)
    assert L.wl_workspace_size(ctypes.byref(s), ctypes.byref(out)) == wl.WL_OK
    small = out.value
    s = _csr(100000, 5000000)
    assert L.wl_workspace_size(ctypes.byref(s), ctypes.byref(out)) == wl.WL_OK
    assert out.value > small
    # linear in n: roughly 60-70 bytes per node plus a little per entry
    assert 40 * 100000 < out.value < 120 * 100000 + 64 * 5000000 // 2048 * 1024


def test_symmetric_flag_adds_the_binned_image_workspace():
    _ensure_built()
    L = wl.lib()
    out = ctypes.c_uint64(0)
    s = _csr(100000, 5000000)
    assert L.wl_workspace_size(ctypes.byref(s), ctypes.byref(out)) == wl.WL_OK
    plain = out.value
    s.flags = wl.WL_CSR_SYMMETRIC
    assert L.wl_workspace_size(ctypes.byref(s), ctypes.byref(out)) == wl.WL_OK
    # 4 bytes per entry of records (one scatter pass at this size) plus tables
    assert plain + 4 * 5000000 <= out.value < plain + 6 * 5000000
    s.weight = 8  # weighted graphs never take that path
    assert L.wl_workspace_size(ctypes.byref(s), ctypes.byref(out)) == wl.WL_OK
    assert out.value == plain


def test_verify_workspace_size_host_only():
    _ensure_built()
    L = wl.lib()
    out = ctypes.c_uint64(0)
    assert L.wl_verify_workspace_size(None, ctypes.byref(out)) == wl.WL_EINVAL
    s = _csr(1000, 5000)
    assert L.wl_verify_workspace_size(ctypes.byref(s), ctypes.byref(out)) == wl.WL_OK
    unweighted = out.value
    # 4 bytes per entry (sorted neighbour colours) plus per-node arrays
    assert 4 * 5000 + 13 * 1000 <= unweighted < 4 * 5000 + 40 * 1000
    s.weight = 8
    assert L.wl_verify_workspace_size(ctypes.byref(s), ctypes.byref(out)) == wl.WL_OK
    assert out.value >= unweighted + 4 * 5000 - 256  # alignment of the regions


def test_host_side_errors():
    _ensure_built()
    L = wl.lib()
    out = ctypes.c_uint64(0)
    assert L.wl_workspace_size(None, ctypes.byref(out)) == wl.WL_EINVAL
    big = _csr(1 << 32, 0)
    assert L.wl_workspace_size(ctypes.byref(big), ctypes.byref(out)) == wl.WL_EOVERFLOW
    assert b"32" in L.wl_last_error()
    # both row pointers set
    s = _csr(10, 20)
    s.row_ptr64 = 8
    k = ctypes.c_uint32(0)
    r = ctypes.c_uint32(0)
    code = L.wl_stable_coloring(ctypes.byref(s), None, 0, 0, ctypes.c_void_p(8),
                                ctypes.byref(k), ctypes.byref(r), ctypes.c_void_p(256),
                                1 << 20, None)
    assert code == wl.WL_EINVAL
    assert b"row_ptr" in L.wl_last_error()
    # NULL outputs
    s = _csr(10, 20)
    assert L.wl_stable_coloring(ctypes.byref(s), None, 0, 0, None, None, None, None, 0,
                                None) == wl.WL_EINVAL
    # k_in out of range in wl_refine_round (checked before any device work)
    code = L.wl_refine_round(ctypes.byref(s), ctypes.c_void_p(8), 0, 0, 0,
                             ctypes.c_void_p(8), ctypes.byref(k), ctypes.c_void_p(256),
                             1 << 20, None)
    assert code == wl.WL_EINVAL
    # workspace too small / misaligned are reported before any device work
    s = _csr(0, 0)
    assert L.wl_stable_coloring(ctypes.byref(s), None, 0, 0, ctypes.c_void_p(8),
                                ctypes.byref(k), ctypes.byref(r), None, 0,
                                None) == wl.WL_OK
    assert k.value == 0 and r.value == 0


def test_binding_refuses_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(wl, "_LIB", None)
    monkeypatch.setattr(wl, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        wl.lib()


def test_precision_setter_is_per_thread_and_checked():
    # host-only calls: no device is touched
    import threading
    assert wl.wl_get_precision() == wl.WL_PRECISION_FP
    with wl.precision(wl.WL_PRECISION_RING64):
        assert wl.wl_get_precision() == 64
        seen = []
        t = threading.Thread(target=lambda: seen.append(wl.wl_get_precision()))
        t.start()
        t.join()
        assert seen == [wl.WL_PRECISION_FP]  # another thread keeps its own
    assert wl.wl_get_precision() == wl.WL_PRECISION_FP
    for bad in (1, 32, 63, 65, 128):
        with pytest.raises(wl.WlError) as e:
            wl.wl_set_precision(bad)
        assert e.value.code == wl.WL_EINVAL
    assert wl.wl_get_precision() == wl.WL_PRECISION_FP


def test_exact_finish_limited_to_verified_size():
    # WL_BATCHED_EXACT is refused above 2^31 entries before any device work
    # (a host-side row pointer array is all the check reads)
    _ensure_built()
    import numpy as np
    L = wl.lib()
    nnz = (1 << 31) + 1
    rp = np.array([0, nnz, nnz], dtype=np.uint64)
    s = wl.WlCsr()
    s.n = 2
    s.nnz = nnz
    s.row_ptr32 = None
    s.row_ptr64 = rp.ctypes.data
    s.col_idx = 16  # never read before the refusal
    s.weight = None
    k, r, o = ctypes.c_uint32(0), ctypes.c_uint32(0), ctypes.c_uint32(0)
    co = ctypes.c_int(0)
    out = np.zeros(2, dtype=np.uint32)
    for opts in (wl.WL_BATCHED_EXACT, wl.WL_BATCHED_EXACT | wl.WL_BATCHED_EARLY_STOP):
        code = L.wl_stable_coloring_batched(ctypes.byref(s), None, 0, 0, opts,
                                            ctypes.c_void_p(out.ctypes.data), ctypes.byref(k),
                                            ctypes.byref(r), ctypes.byref(o), ctypes.byref(co),
                                            ctypes.c_void_p(256), 1 << 30, None)
        assert code == wl.WL_EINVAL
        assert b"2^31" in L.wl_last_error()


def test_noalloc_refuses_graphs_beyond_its_scratch():
    # the size check comes before any device work
    _ensure_built()
    L = wl.lib()
    s = _csr(2_000_000, 0, rp32=False)
    k, r = ctypes.c_uint32(0), ctypes.c_uint32(0)
    code = L.wl_stable_coloring_noalloc(ctypes.byref(s), None, 0, 0, ctypes.c_void_p(256),
                                        ctypes.byref(k), ctypes.byref(r), None)
    assert code == wl.WL_EBUDGET
    assert b"scratch" in L.wl_last_error()
    need = ctypes.c_uint64(0)
    assert L.wl_workspace_size(ctypes.byref(s), ctypes.byref(need)) == wl.WL_OK
    assert need.value > wl.WL_NOALLOC_SCRATCH_BYTES
    # an empty graph needs nothing
    s = _csr(0, 0)
    assert L.wl_stable_coloring_noalloc(ctypes.byref(s), None, 0, 0, None, ctypes.byref(k),
                                        ctypes.byref(r), None) == wl.WL_OK
