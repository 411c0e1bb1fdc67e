"""Seeded synthetic graph inputs (undirected graphs stored as symmetric CSR).

This module holds only input generation.  It is shared by the tests, the
benchmark and the oracle side; it contains nothing of the colour-refinement
arithmetic.  Every random number is a counter-based SplitMix64 output
(``gen_common.h``), so the CPU and GPU builds produce identical graphs; the
CSR of a simple graph with sorted rows is canonical, so "identical" is
checked byte for byte.

Workloads (the paper's datasets are not available; these stand in for them):

* ``er_graph``      Erdos-Renyi G(n, m): first m distinct pairs of the stream.
* ``grid_graph``    a x b 4-neighbour grid, id = r * b + s, no wrap-around.
* ``chung_lu``      power-law graph by edge sampling, weights (i+1)^(-1/(g-1)).
* ``rmat``          R-MAT with Graph500 parameters and a seeded vertex
                    bijection; self-loops dropped, symmetrised, deduplicated.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_CPU = None
_GPU = None
MAX64 = np.uint64(0xFFFFFFFFFFFFFFFF)


class CSR:
    """n nodes; row_ptr (n+1), col (nnz, uint32) as numpy or torch arrays."""

    def __init__(self, n, row_ptr, col, weight=None, name=""):
        self.n = int(n)
        self.row_ptr = row_ptr
        self.col = col
        self.weight = weight
        self.name = name

    @property
    def nnz(self):
        return int(self.col.shape[0])

    def degrees(self):
        rp = self.row_ptr
        return rp[1:] - rp[:-1]

    def to_numpy(self):
        if isinstance(self.row_ptr, np.ndarray):
            return self
        w = None if self.weight is None else self.weight.cpu().numpy()
        return CSR(self.n, self.row_ptr.cpu().numpy(), self.col.cpu().numpy(), w,
                   self.name)


def _cpu():
    global _CPU
    if _CPU is None:
        path = os.path.join(_HERE, "libwlgen_cpu.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: run python -m paper_2607_02603_amd.build")
        lib = ctypes.CDLL(path)
        u64, u32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p
        lib.gen_rmat_keys_cpu.argtypes = [u32, u64, u64, u64, u32, u32, u32, vp]
        lib.gen_rmat_keys_cpu.restype = None
        lib.gen_chunglu_keys_cpu.argtypes = [u32, u64, u64, u64, vp, vp, vp]
        lib.gen_chunglu_keys_cpu.restype = None
        lib.gen_alias_build.argtypes = [u32, vp, vp, vp]
        lib.gen_alias_build.restype = ctypes.c_int
        lib.gen_er_edges.argtypes = [u32, u64, u64, vp, vp]
        lib.gen_er_edges.restype = u64
        _CPU = lib
    return _CPU


def _gpu():
    global _GPU
    if _GPU is None:
        path = os.path.join(_HERE, "libwlgen_gpu.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: run python -m paper_2607_02603_amd.build")
        lib = ctypes.CDLL(path)
        u64, u32, vp, i32 = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_int
        lib.gen_rmat_gpu.argtypes = [i32, u32, u64, u32, u32, u32, u64, u64, u32, u32,
                                     vp, vp, vp]
        lib.gen_rmat_gpu.restype = i32
        lib.gen_chunglu_gpu.argtypes = [i32, u32, u64, vp, vp, u64, u64, u32, u32, vp,
                                        vp, vp]
        lib.gen_chunglu_gpu.restype = i32
        _GPU = lib
    return _GPU


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def csr_from_keys(keys, n, name=""):
    """Directed-entry keys (u << 32 | v, UINT64_MAX = none) -> CSR with sorted,
    deduplicated rows.  row_ptr is uint32 when nnz < 2^32, else uint64."""
    keys = keys[keys != MAX64]
    keys = np.unique(keys)
    u = (keys >> np.uint64(32)).astype(np.int64)
    v = (keys & np.uint64(0xFFFFFFFF)).astype(np.uint32)
    cnt = np.bincount(u, minlength=n).astype(np.uint64)
    rp = np.zeros(n + 1, dtype=np.uint64)
    np.cumsum(cnt, out=rp[1:])
    if v.size < 2**32:
        rp = rp.astype(np.uint32)
    return CSR(n, rp, v, None, name)


def csr_from_edges(n, u, v, name=""):
    """Undirected edge list -> symmetric simple CSR (self-loops dropped)."""
    u = np.asarray(u, dtype=np.uint64)
    v = np.asarray(v, dtype=np.uint64)
    keep = u != v
    u, v = u[keep], v[keep]
    keys = np.concatenate([(u << np.uint64(32)) | v, (v << np.uint64(32)) | u])
    return csr_from_keys(keys, n, name)


# ---------------------------------------------------------------------------
# Configurations
# ---------------------------------------------------------------------------

def er_graph(n=20000, m=80000, seed=0):
    """G(n, m): the first m distinct unordered pairs u != v of the stream."""
    u = np.empty(m, dtype=np.uint32)
    v = np.empty(m, dtype=np.uint32)
    _cpu().gen_er_edges(n, m, seed, _ptr(u), _ptr(v))
    return csr_from_edges(n, u, v, name=f"er_n{n}_m{m}_s{seed}")


def grid_graph(a=1024, b=None):
    """a x b grid, 4-neighbour, id = r * b + s, no wrap-around."""
    b = a if b is None else b
    ids = np.arange(a * b, dtype=np.uint64).reshape(a, b)
    hu, hv = ids[:, :-1].ravel(), ids[:, 1:].ravel()
    vu, vv = ids[:-1, :].ravel(), ids[1:, :].ravel()
    return csr_from_edges(a * b, np.concatenate([hu, vu]), np.concatenate([hv, vv]),
                          name=f"grid_{a}x{b}")


def chung_lu_alias(n, gamma=2.1):
    """Alias table of w_i = (i + 1)^(-1/(gamma - 1)) (built on the host)."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-1.0 / (gamma - 1.0))
    thr = np.empty(n, dtype=np.uint64)
    alias = np.empty(n, dtype=np.uint32)
    if _cpu().gen_alias_build(n, _ptr(w), _ptr(thr), _ptr(alias)) != 0:
        raise MemoryError("alias table")
    return thr, alias


def _bucket_plan(n_nodes_pow2_bits, total_keys, max_per_bucket=1 << 27):
    bits = 0
    while (total_keys >> bits) > max_per_bucket and bits < 10:
        bits += 1
    bits = min(bits, n_nodes_pow2_bits)
    return bits


def chung_lu(n=4_000_000, samples=64_000_000, gamma=2.1, seed=0, device="cpu"):
    """Chung-Lu power-law graph by edge sampling (both endpoints drawn
    proportionally to w_i = (i+1)^(-1/(gamma-1))), symmetrised, deduplicated."""
    thr, alias = chung_lu_alias(n, gamma)
    name = f"chunglu_n{n}_s{samples}_g{gamma}_s{seed}"
    if device == "cpu":
        keys = np.empty(2 * samples, dtype=np.uint64)
        _cpu().gen_chunglu_keys_cpu(n, 0, samples, seed, _ptr(thr), _ptr(alias),
                                    _ptr(keys))
        return csr_from_keys(keys, n, name)
    import torch
    dthr = torch.from_numpy(thr.view(np.int64)).to(device)
    dal = torch.from_numpy(alias.view(np.int32)).to(device)
    nbits = max(1, int(np.ceil(np.log2(n))))

    def emit(phase, shift, nbk, arr, keys, stream):
        return _gpu().gen_chunglu_gpu(phase, n, seed, dthr.data_ptr(), dal.data_ptr(),
                                      0, samples, shift, nbk, arr, keys, stream)
    return _gpu_build(n, nbits, 2 * samples, emit, name, device)


def rmat_thresholds(abcd):
    a, b, c, _ = abcd
    t = lambda x: min(int(x * 4294967296.0), 0xFFFFFFFF)  # noqa: E731
    return t(a), t(a + b), t(a + b + c)


def rmat(scale=27, edge_factor=16, abcd=(0.57, 0.19, 0.19, 0.05), seed=0,
         device="cpu"):
    """R-MAT, edge_factor * 2^scale samples, seeded vertex bijection, self-loops
    dropped, symmetrised, deduplicated."""
    n = 1 << scale
    samples = edge_factor * n
    ta, tab, tabc = rmat_thresholds(abcd)
    name = f"rmat_s{scale}_ef{edge_factor}_s{seed}"
    if device == "cpu":
        keys = np.empty(2 * samples, dtype=np.uint64)
        _cpu().gen_rmat_keys_cpu(scale, 0, samples, seed, ta, tab, tabc, _ptr(keys))
        return csr_from_keys(keys, n, name)

    def emit(phase, shift, nbk, arr, keys, stream):
        return _gpu().gen_rmat_gpu(phase, scale, seed, ta, tab, tabc, 0, samples, shift,
                                   nbk, arr, keys, stream)
    return _gpu_build(n, scale, 2 * samples, emit, name, device)


def _gpu_build(n, nbits, max_keys, emit, name, device):
    """Bucketed generation on the GPU: count, scatter, then per bucket sort +
    unique + row counts (torch ops).  Returns a CSR of torch tensors on
    'device' with row_ptr int64 (uint64 values) and col int32 (uint32 values)."""
    import torch
    bbits = _bucket_plan(nbits, max_keys)
    nbk = 1 << bbits
    shift = nbits - bbits
    stream = torch.cuda.current_stream(device).cuda_stream
    counts = torch.zeros(nbk, dtype=torch.int64, device=device)
    if emit(0, shift, nbk, counts.data_ptr(), 0, stream) != 0:
        raise RuntimeError("graph generator count pass failed")
    offs = torch.zeros(nbk + 1, dtype=torch.int64, device=device)
    offs[1:] = torch.cumsum(counts, 0)
    total = int(offs[-1].item())
    keys = torch.empty(max(total, 1), dtype=torch.int64, device=device)
    cursor = offs[:-1].clone()
    if emit(1, shift, nbk, cursor.data_ptr(), keys.data_ptr(), stream) != 0:
        raise RuntimeError("graph generator scatter pass failed")
    offs_h = offs.cpu().tolist()
    rows_per = 1 << shift
    row_cnt = torch.zeros(n, dtype=torch.int64, device=device)
    cols = []
    for b in range(nbk):
        seg = keys[offs_h[b]:offs_h[b + 1]]
        if seg.numel() == 0:
            continue
        seg = torch.sort(seg).values
        seg = torch.unique_consecutive(seg)
        u = seg >> 32
        lo = b * rows_per
        hi = min(n, lo + rows_per)
        row_cnt[lo:hi] = torch.bincount(u - lo, minlength=hi - lo)
        cols.append((seg & 0xFFFFFFFF).to(torch.int32))
        del seg, u
    del keys
    col = torch.cat(cols) if cols else torch.empty(0, dtype=torch.int32, device=device)
    del cols
    rp = torch.zeros(n + 1, dtype=torch.int64, device=device)
    rp[1:] = torch.cumsum(row_cnt, 0)
    return CSR(n, rp, col, None, name)
