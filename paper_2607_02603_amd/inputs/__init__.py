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
                                     u32, u32, vp, vp, vp]
        lib.gen_rmat_gpu.restype = i32
        lib.gen_chunglu_gpu.argtypes = [i32, u32, u64, vp, vp, u64, u64, u32, u32, u32,
                                        u32, vp, vp, vp]
        lib.gen_chunglu_gpu.restype = i32
        lib.gen_host_alloc.argtypes = [u64]
        lib.gen_host_alloc.restype = vp
        lib.gen_host_free.argtypes = [vp]
        lib.gen_host_free.restype = None
        _GPU = lib
    return _GPU


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


class _PinnedOwner:
    def __init__(self, ptr):
        self.ptr = ptr

    def __del__(self):
        if self.ptr and _GPU is not None:
            _GPU.gen_host_free(self.ptr)
            self.ptr = None


def pinned_empty(count, dtype):
    """A torch tensor of 'count' elements in pinned host memory of exactly
    that size (torch's own pinned allocator rounds up to powers of two)."""
    import torch
    np_dtype = {torch.int32: np.int32, torch.int64: np.int64,
                torch.uint8: np.uint8}[dtype]
    nbytes = max(int(count), 1) * np.dtype(np_dtype).itemsize
    ptr = _gpu().gen_host_alloc(nbytes)
    if not ptr:
        raise MemoryError(f"hipHostMalloc({nbytes}) failed")
    buf = (ctypes.c_char * nbytes).from_address(ptr)
    # the buffer object frees the allocation when the last view of it dies:
    # numpy keeps the buffer alive, torch keeps the numpy array alive
    buf._wl_owner = _PinnedOwner(ptr)
    arr = np.frombuffer(buf, dtype=np_dtype, count=max(int(count), 1))
    t = torch.from_numpy(arr)
    return t if count else t[:0]


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

    def emit(phase, shift, nbk, blo, bhi, arr, keys, stream):
        return _gpu().gen_chunglu_gpu(phase, n, seed, dthr.data_ptr(), dal.data_ptr(),
                                      0, samples, shift, nbk, blo, bhi, arr, keys, stream)
    return _gpu_build(n, nbits, 2 * samples, emit, name, device)


def rmat_thresholds(abcd):
    a, b, c, _ = abcd
    t = lambda x: min(int(x * 4294967296.0), 0xFFFFFFFF)  # noqa: E731
    return t(a), t(a + b), t(a + b + c)


def rmat(scale=27, edge_factor=16, abcd=(0.57, 0.19, 0.19, 0.05), seed=0,
         device="cpu", host_out=False, directed=False, pinned=True):
    """R-MAT, edge_factor * 2^scale samples, seeded vertex bijection, self-loops
    dropped, symmetrised, deduplicated.  device='cuda' generates on the GPU;
    with host_out=True the CSR is returned in pinned host memory and the
    device never holds more than a group of buckets (for graphs larger than
    HBM; pinned=False puts it in pageable memory instead, for graphs larger
    than the page-locked memory a process may hold).  directed=True (host
    generation only) keeps each sample as the one
    entry u -> v, as for a web graph: out- and in-degrees are both skewed and
    many nodes have no out-edge."""
    n = 1 << scale
    samples = edge_factor * n
    ta, tab, tabc = rmat_thresholds(abcd)
    name = f"rmat_s{scale}_ef{edge_factor}_s{seed}" + ("_dir" if directed else "")
    if device == "cpu":
        keys = np.empty(2 * samples, dtype=np.uint64)
        _cpu().gen_rmat_keys_cpu(scale, 0, samples, seed, ta, tab, tabc, _ptr(keys))
        if directed:
            keys = keys[0::2]  # the entry u -> v of every sample (see gen_cpu.c)
        return csr_from_keys(keys, n, name)
    if directed:
        raise ValueError("directed R-MAT is generated on the host only")

    def emit(phase, shift, nbk, blo, bhi, arr, keys, stream):
        return _gpu().gen_rmat_gpu(phase, scale, seed, ta, tab, tabc, 0, samples, shift,
                                   nbk, blo, bhi, arr, keys, stream)
    return _gpu_build(n, scale, 2 * samples, emit, name, device, host_out, pinned=pinned)


def _gpu_build(n, nbits, max_keys, emit, name, device, host_out=False,
               group_keys=1 << 31, pinned=True):
    """Bucketed generation on the GPU: count, then per group of buckets
    scatter + per bucket sort + unique + row counts (torch ops).  Returns a
    CSR with row_ptr int64 (uint64 values) and col int32 (uint32 values), on
    'device' or, with host_out, in pinned host memory."""
    import torch
    bbits = _bucket_plan(nbits, max_keys)
    nbk = 1 << bbits
    shift = nbits - bbits
    stream = torch.cuda.current_stream(device).cuda_stream
    counts = torch.zeros(nbk, dtype=torch.int64, device=device)
    if emit(0, shift, nbk, 0, nbk, counts.data_ptr(), 0, stream) != 0:
        raise RuntimeError("graph generator count pass failed")
    cnt_h = counts.cpu().tolist()
    total = sum(cnt_h)
    if not host_out:
        group_keys = max(total, 1)
    rows_per = 1 << shift
    row_cnt = torch.zeros(n, dtype=torch.int64, device=device)
    cols = []
    pos = 0
    b0 = 0
    while b0 < nbk:
        b1, gk = b0, 0
        while b1 < nbk and (b1 == b0 or gk + cnt_h[b1] <= group_keys):
            gk += cnt_h[b1]
            b1 += 1
        keys = torch.empty(max(gk, 1), dtype=torch.int64, device=device)
        cur = [0] * nbk
        acc = 0
        for b in range(b0, b1):
            cur[b] = acc
            acc += cnt_h[b]
        cursor = torch.tensor(cur, dtype=torch.int64, device=device)
        if emit(1, shift, nbk, b0, b1, cursor.data_ptr(), keys.data_ptr(), stream) != 0:
            raise RuntimeError("graph generator scatter pass failed")
        for b in range(b0, b1):
            seg = keys[cur[b]:cur[b] + cnt_h[b]]
            if seg.numel() == 0:
                continue
            seg = torch.sort(seg).values
            seg = torch.unique_consecutive(seg)
            u = seg >> 32
            lo = b * rows_per
            hi = min(n, lo + rows_per)
            row_cnt[lo:hi] = torch.bincount(u - lo, minlength=hi - lo)
            c = (seg & 0xFFFFFFFF).to(torch.int32)
            cols.append(c)
            pos += c.numel()
            del seg, u, c
        del keys
        b0 = b1
    rp = torch.zeros(n + 1, dtype=torch.int64, device=device)
    rp[1:] = torch.cumsum(row_cnt, 0)
    if host_out:
        # page-locked memory is capped per process: take exactly nnz entries
        del row_cnt
        alloc = pinned_empty if pinned else (lambda c, dt: torch.empty(c, dtype=dt))
        rp_h = alloc(n + 1, torch.int64)
        rp_h.copy_(rp)
        del rp
        col_h = alloc(pos, torch.int32)
        at = 0
        for c in cols:
            col_h[at:at + c.numel()].copy_(c)
            at += c.numel()
        del cols
        return CSR(n, rp_h, col_h, None, name)
    col = torch.cat(cols) if cols else torch.empty(0, dtype=torch.int32, device=device)
    del cols
    return CSR(n, rp, col, None, name)
