"""Randomized 1-WL stable colouring on MI355X (gfx950).

Thin Python binding over the C ABI of ``include/wl.h`` (``libwl.so``, built
in-tree by ``python -m paper_2607_02603_amd.build``).  The functions have the
same names as the C entry points and only marshal arguments: every step of
the method runs in the library's HIP kernels.  PyTorch provides device
memory (tensors) and the stream (the current HIP stream).

There is no CPU fallback: if the library is missing, importing the binding
works but every call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwl.so")

WL_OK = 0
WL_EINVAL = -1
WL_EBUDGET = -2
WL_EOVERFLOW = -3
WL_EMAXROUNDS = -4
WL_ENOTSTABLE = -5
WL_EHIP = -6
WL_ENOMEM = -7
_NAMES = {-1: "WL_EINVAL", -2: "WL_EBUDGET", -3: "WL_EOVERFLOW",
          -4: "WL_EMAXROUNDS", -5: "WL_ENOTSTABLE", -6: "WL_EHIP", -7: "WL_ENOMEM"}

EXPORTED = ["wl_workspace_size", "wl_batched_workspace_size", "wl_refine_round",
            "wl_stable_coloring", "wl_stable_coloring_batched", "wl_streamed_workspace_size",
            "wl_stable_coloring_streamed", "wl_verify_workspace_size", "wl_verify_stable",
            "wl_stats_enable", "wl_stats_get", "wl_set_precision", "wl_get_precision",
            "wl_stable_coloring_noalloc", "wl_last_error"]

WL_NOALLOC_SCRATCH_BYTES = 64 << 20

WL_STATS_TIME = 1
WL_STATS_WORK = 2

WL_BATCHED_EXACT = 1
WL_BATCHED_EARLY_STOP = 2

WL_PRECISION_FP = 0
WL_PRECISION_RING64 = 64


class WlError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{_NAMES.get(code, code)}: {msg}")
        self.code = code


class WlStatsKind(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_uint32), ("pad", ctypes.c_uint32),
                ("ms", ctypes.c_double), ("rows", ctypes.c_uint64),
                ("entries", ctypes.c_uint64)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "pad"}


class WlStats(ctypes.Structure):
    _fields_ = [("rounds", ctypes.c_uint32), ("pad", ctypes.c_uint32),
                ("call_ms", ctypes.c_double), ("gather", WlStatsKind),
                ("pb", WlStatsKind), ("uniform", WlStatsKind)]

    def as_dict(self):
        return {"rounds": self.rounds, "call_ms": self.call_ms,
                "gather": self.gather.as_dict(), "pb": self.pb.as_dict(),
                "uniform": self.uniform.as_dict()}


WL_CSR_SYMMETRIC = 1


class WlCsr(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint64), ("nnz", ctypes.c_uint64),
                ("row_ptr32", ctypes.c_void_p), ("row_ptr64", ctypes.c_void_p),
                ("col_idx", ctypes.c_void_p), ("weight", ctypes.c_void_p),
                ("flags", ctypes.c_uint64)]


_LIB = None


def lib():
    """The loaded libwl.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with "
                               "`python -m paper_2607_02603_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, u64, u32, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int
        P = ctypes.POINTER
        L.wl_workspace_size.argtypes = [P(WlCsr), P(u64)]
        L.wl_batched_workspace_size.argtypes = [P(WlCsr), u64, P(u64)]
        L.wl_refine_round.argtypes = [P(WlCsr), vp, u32, u64, u32, vp, P(u32), vp, u64, vp]
        L.wl_stable_coloring.argtypes = [P(WlCsr), vp, u64, u32, vp, P(u32), P(u32), vp,
                                         u64, vp]
        L.wl_stable_coloring_noalloc.argtypes = [P(WlCsr), vp, u64, u32, vp, P(u32), P(u32),
                                                 vp]
        L.wl_stable_coloring_batched.argtypes = [P(WlCsr), vp, u64, u64, u32, vp, P(u32),
                                                 P(u32), P(u32), P(i32), vp, u64, vp]
        L.wl_streamed_workspace_size.argtypes = [P(WlCsr), P(u64)]
        L.wl_stable_coloring_streamed.argtypes = [P(WlCsr), vp, u64, u32, vp, P(u32), P(u32),
                                                  vp, u64, vp]
        L.wl_verify_workspace_size.argtypes = [P(WlCsr), P(u64)]
        L.wl_verify_stable.argtypes = [P(WlCsr), vp, u32, vp, u64, vp]
        L.wl_stats_enable.argtypes = [i32]
        L.wl_stats_get.argtypes = [P(WlStats)]
        L.wl_set_precision.argtypes = [u32]
        L.wl_get_precision.argtypes = [P(u32)]
        L.wl_last_error.restype = ctypes.c_char_p
        for f in EXPORTED[:-1]:
            getattr(L, f).restype = i32
        _LIB = L
    return _LIB


def _check(code):
    if code != WL_OK:
        raise WlError(code, lib().wl_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


class Graph:
    """CSR adjacency whose arrays live in torch tensors (device or host).

    row_ptr: int32/int64 tensor of n+1 entries (values read as uint32/uint64);
    col_idx: int32 tensor (uint32 values); weight: None or int32 (uint32);
    symmetric: the caller states that A equals its transpose (WL_CSR_SYMMETRIC).
    """

    def __init__(self, n, row_ptr, col_idx, weight=None, symmetric=False):
        self.n = int(n)
        self.symmetric = bool(symmetric)
        self.row_ptr = row_ptr.contiguous()
        self.col_idx = col_idx.contiguous()
        self.weight = None if weight is None else weight.contiguous()
        if self.row_ptr.dtype not in (torch.int32, torch.int64):
            raise TypeError("row_ptr must be int32 or int64")
        if self.col_idx.dtype != torch.int32:
            raise TypeError("col_idx must be int32")
        if self.weight is not None and self.weight.dtype != torch.int32:
            raise TypeError("weight must be int32")
        if self.row_ptr.numel() != self.n + 1:
            raise ValueError("row_ptr must have n+1 entries")

    @property
    def nnz(self):
        return int(self.col_idx.numel())

    @property
    def device(self):
        return self.col_idx.device

    def csr(self):
        s = WlCsr()
        s.n = self.n
        s.nnz = self.nnz
        rp = self.row_ptr.data_ptr()
        s.row_ptr32 = rp if self.row_ptr.dtype == torch.int32 else None
        s.row_ptr64 = rp if self.row_ptr.dtype == torch.int64 else None
        s.col_idx = self.col_idx.data_ptr() if self.nnz else None
        s.weight = None if self.weight is None else self.weight.data_ptr()
        s.flags = WL_CSR_SYMMETRIC if self.symmetric else 0
        return s

    @classmethod
    def from_numpy(cls, n, row_ptr, col, weight=None, device="cuda", symmetric=False):
        import numpy as np
        rp = np.ascontiguousarray(row_ptr)
        if rp.dtype in (np.uint64, np.int64):
            rp_t = torch.from_numpy(rp.view(np.int64))
        else:
            rp_t = torch.from_numpy(rp.astype(np.uint32).view(np.int32))
        col_t = torch.from_numpy(np.asarray(col, dtype=np.uint32).view(np.int32))
        w_t = None if weight is None else torch.from_numpy(
            np.asarray(weight, dtype=np.uint32).view(np.int32))
        if device is not None:
            rp_t, col_t = rp_t.to(device), col_t.to(device)
            w_t = None if w_t is None else w_t.to(device)
        return cls(n, rp_t, col_t, w_t, symmetric)


def wl_workspace_size(g):
    out = ctypes.c_uint64(0)
    s = g.csr()
    _check(lib().wl_workspace_size(ctypes.byref(s), ctypes.byref(out)))
    return int(out.value)


def wl_batched_workspace_size(g, max_batch_entries=0):
    out = ctypes.c_uint64(0)
    s = g.csr()
    _check(lib().wl_batched_workspace_size(ctypes.byref(s), max_batch_entries,
                                           ctypes.byref(out)))
    return int(out.value)


def workspace(nbytes, device="cuda"):
    """A device byte buffer usable as workspace (256-byte aligned)."""
    buf = torch.empty(max(int(nbytes), 1) + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf[off:off + max(int(nbytes), 1)]


def _ws(g, ws):
    if ws is None:
        ws = workspace(wl_workspace_size(g), g.device)
    return ws


def wl_refine_round(g, color_in, k_in, seed, round_, color_out=None, ws=None,
                    stream=None):
    """One round of Algorithm 1.  Returns (color_out, k_out)."""
    ws = _ws(g, ws)
    if color_out is None:
        color_out = torch.empty(g.n, dtype=torch.int32, device=g.device)
    k = ctypes.c_uint32(0)
    s = g.csr()
    _check(lib().wl_refine_round(ctypes.byref(s), _ptr(color_in), k_in, seed, round_,
                                 _ptr(color_out), ctypes.byref(k), _ptr(ws),
                                 ws.numel(), _stream(stream)))
    return color_out, int(k.value)


def wl_stable_coloring(g, init_color=None, seed=0, max_rounds=0, color_out=None,
                       ws=None, stream=None, allow_max_rounds=False):
    """Algorithm 1 to completion.  Returns (colors, k, rounds).  With
    allow_max_rounds=True a WL_EMAXROUNDS result is returned instead of
    raised (the colours are then those of the last round)."""
    ws = _ws(g, ws)
    if color_out is None:
        color_out = torch.empty(g.n, dtype=torch.int32, device=g.device)
    k = ctypes.c_uint32(0)
    r = ctypes.c_uint32(0)
    s = g.csr()
    code = lib().wl_stable_coloring(ctypes.byref(s), _ptr(init_color), seed, max_rounds,
                                    _ptr(color_out), ctypes.byref(k), ctypes.byref(r),
                                    _ptr(ws), ws.numel(), _stream(stream))
    if not (allow_max_rounds and code == WL_EMAXROUNDS):
        _check(code)
    return color_out, int(k.value), int(r.value)


def wl_stable_coloring_noalloc(g, init_color=None, seed=0, max_rounds=0, color_out=None,
                               stream=None):
    """Algorithm 1 to completion without a workspace (the library's fixed
    per-GPU scratch of WL_NOALLOC_SCRATCH_BYTES).  Returns (colors, k,
    rounds).  Only the output array is allocated here, and only when
    color_out is None."""
    if color_out is None:
        color_out = torch.empty(g.n, dtype=torch.int32, device=g.device)
    k = ctypes.c_uint32(0)
    r = ctypes.c_uint32(0)
    s = g.csr()
    _check(lib().wl_stable_coloring_noalloc(ctypes.byref(s), _ptr(init_color), seed,
                                            max_rounds, _ptr(color_out), ctypes.byref(k),
                                            ctypes.byref(r), _stream(stream)))
    return color_out, int(k.value), int(r.value)


def wl_stable_coloring_batched(g_host, init_host=None, seed=0, max_batch_entries=0,
                               ws=None, ws_bytes=None, device="cuda", stream=None,
                               options=0):
    """Algorithm 2.  g_host: Graph with host tensors (pinned recommended).
    options: WL_BATCHED_EXACT and / or WL_BATCHED_EARLY_STOP.
    Returns (colors (host int32), k, rounds, outer, coarsest)."""
    if ws is None:
        cap = min(max_batch_entries, max(g_host.nnz, 1)) if max_batch_entries else 0
        nb = ws_bytes or wl_batched_workspace_size(g_host, cap)
        if options & WL_BATCHED_EXACT and not ws_bytes:
            nb = max(nb, wl_streamed_workspace_size(g_host))
        ws = workspace(nb, device)
    out = torch.empty(g_host.n, dtype=torch.int32)
    k, r, o = ctypes.c_uint32(0), ctypes.c_uint32(0), ctypes.c_uint32(0)
    co = ctypes.c_int(0)
    s = g_host.csr()
    _check(lib().wl_stable_coloring_batched(
        ctypes.byref(s), _ptr(init_host), seed, max_batch_entries, options, _ptr(out),
        ctypes.byref(k), ctypes.byref(r), ctypes.byref(o), ctypes.byref(co), _ptr(ws),
        ws.numel(), _stream(stream)))
    return out, int(k.value), int(r.value), int(o.value), bool(co.value)


def wl_streamed_workspace_size(g):
    out = ctypes.c_uint64(0)
    s = g.csr()
    _check(lib().wl_streamed_workspace_size(ctypes.byref(s), ctypes.byref(out)))
    return int(out.value)


def wl_stable_coloring_streamed(g_host, init_host=None, seed=0, max_rounds=0, ws=None,
                                ws_bytes=None, device="cuda", stream=None,
                                allow_max_rounds=False):
    """Algorithm 1 with the entries in host memory (streamed image).
    Returns (colors (host int32), k, rounds); same ids as wl_stable_coloring."""
    if ws is None:
        ws = workspace(ws_bytes or wl_streamed_workspace_size(g_host), device)
    out = torch.empty(g_host.n, dtype=torch.int32)
    k, r = ctypes.c_uint32(0), ctypes.c_uint32(0)
    s = g_host.csr()
    code = lib().wl_stable_coloring_streamed(
        ctypes.byref(s), _ptr(init_host), seed, max_rounds, _ptr(out), ctypes.byref(k),
        ctypes.byref(r), _ptr(ws), ws.numel(), _stream(stream))
    if not (allow_max_rounds and code == WL_EMAXROUNDS):
        _check(code)
    return out, int(k.value), int(r.value)


def wl_verify_workspace_size(g):
    out = ctypes.c_uint64(0)
    s = g.csr()
    _check(lib().wl_verify_workspace_size(ctypes.byref(s), ctypes.byref(out)))
    return int(out.value)


def wl_verify_stable(g, color, k, ws=None, stream=None):
    """True if the colouring is stable (exact certificate), else False."""
    if ws is None:
        ws = workspace(wl_verify_workspace_size(g), g.device)
    s = g.csr()
    code = lib().wl_verify_stable(ctypes.byref(s), _ptr(color), k, _ptr(ws), ws.numel(),
                                  _stream(stream))
    if code == WL_ENOTSTABLE:
        return False
    _check(code)
    return True


def wl_set_precision(q):
    """Arithmetic of the image step for this thread's later calls:
    WL_PRECISION_FP (0, F_p with p = 2^61 - 1) or WL_PRECISION_RING64 (64,
    the ring Z/2^64 of Algorithm 1 with q = 64)."""
    _check(lib().wl_set_precision(q))


def wl_get_precision():
    out = ctypes.c_uint32(0)
    _check(lib().wl_get_precision(ctypes.byref(out)))
    return int(out.value)


class precision:
    """Context manager: ``with precision(WL_PRECISION_RING64): ...`` runs the
    block's calls (on this thread) in that arithmetic and restores the
    previous one."""

    def __init__(self, q):
        self.q = q
        self.prev = None

    def __enter__(self):
        self.prev = wl_get_precision()
        wl_set_precision(self.q)
        return self

    def __exit__(self, *exc):
        wl_set_precision(self.prev)
        return False


def wl_stats_enable(flags):
    """Turn diagnostics on for this thread (WL_STATS_TIME | WL_STATS_WORK)."""
    _check(lib().wl_stats_enable(flags))


def wl_stats_get():
    """Diagnostics of the last in-core call on this thread, as a dict:
    rounds, call_ms and, per image kind ('gather', 'pb', 'uniform'), the
    launches, their summed ms, and the rows and entries they read."""
    st = WlStats()
    _check(lib().wl_stats_get(ctypes.byref(st)))
    return st.as_dict()
