"""CPU oracle for randomized 1-WL stable colouring — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never imports it, and the two share no code.

Thin ctypes wrapper over ``oracle/wl_oracle.c`` (plain C, 128-bit exact sums,
qsort-based relabel; Algorithm 1, classic refinement, splitter-based exact
refinement and Algorithm 2) plus pure-Python pieces for tiny inputs
(``oracle.bruteforce``).  Section, equation and algorithm names refer to
"Scaling Weisfeiler-Leman Expressiveness Analysis to Massive Graphs with
GPUs".

Parity status of each function is recorded in its docstring; every function
here is pinned by ``tests/test_oracle_*.py`` against brute force, closed
forms, automorphism orbits or published SplitMix64 outputs.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

P61 = (1 << 61) - 1
GAMMA = 0x9E3779B97F4A7C15

# Arithmetic of the image step (argument q): F_p with p = 2^61 - 1, or the
# ring Z/2^64 of Section 4.1 (Algorithm 1 with precision q = 64).
FP = 0
RING64 = 64


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "liboracle.so")
        src = os.path.join(_HERE, "wl_oracle.c")
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(src):
            from . import build as _b  # noqa: F401  (oracle/build.py)
            _b.build()
        lib = ctypes.CDLL(path)
        u64, u32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p
        lib.orc_mix64.restype = u64
        lib.orc_mix64.argtypes = [u64]
        lib.orc_splitmix_nth.restype = u64
        lib.orc_splitmix_nth.argtypes = [u64, u64]
        lib.orc_round_key.restype = u64
        lib.orc_round_key.argtypes = [u64, u64]
        lib.orc_weight.restype = u64
        lib.orc_weight.argtypes = [u64, u64, u64]
        lib.orc_weight_q.restype = u64
        lib.orc_weight_q.argtypes = [u64, u64, u64, u32]
        lib.orc_ring_preconditions.restype = ctypes.c_int
        lib.orc_ring_preconditions.argtypes = [u64, vp, vp]
        lib.orc_canonicalize.restype = u32
        lib.orc_canonicalize.argtypes = [u64, vp, vp]
        lib.orc_image.restype = None
        lib.orc_image.argtypes = [u64, vp, vp, vp, vp, u32, u64, u64, vp]
        lib.orc_image_q.restype = ctypes.c_int
        lib.orc_image_q.argtypes = [u64, vp, vp, vp, vp, u32, u64, u64, vp, u32]
        lib.orc_relabel.restype = u32
        lib.orc_relabel.argtypes = [u64, vp, vp, vp]
        lib.orc_refine_round.restype = u32
        lib.orc_refine_round.argtypes = [u64, vp, vp, vp, vp, u32, u64, u64, vp, vp]
        lib.orc_refine_round_q.restype = u32
        lib.orc_refine_round_q.argtypes = [u64, vp, vp, vp, vp, u32, u64, u64, vp, vp, u32]
        lib.orc_stable_coloring.restype = ctypes.c_int
        lib.orc_stable_coloring.argtypes = [u64, vp, vp, vp, vp, u64, u32, vp, vp, vp, vp]
        lib.orc_stable_coloring_q.restype = ctypes.c_int
        lib.orc_stable_coloring_q.argtypes = [u64, vp, vp, vp, vp, u64, u32, vp, vp, vp, vp,
                                              u32]
        lib.orc_classic_round.restype = u32
        lib.orc_classic_round.argtypes = [u64, vp, vp, vp, vp, vp]
        lib.orc_classic_coloring.restype = ctypes.c_int
        lib.orc_classic_coloring.argtypes = [u64, vp, vp, vp, vp, u32, vp, vp, vp, vp]
        lib.orc_splitter_coloring.restype = ctypes.c_int
        lib.orc_splitter_coloring.argtypes = [u64, vp, vp, vp, vp, vp, vp, vp]
        lib.orc_is_stable.restype = ctypes.c_int
        lib.orc_is_stable.argtypes = [u64, vp, vp, vp, vp, u32]
        lib.orc_first_occurrence.restype = u32
        lib.orc_first_occurrence.argtypes = [u64, vp, vp]
        lib.orc_batch_cut.restype = u64
        lib.orc_batch_cut.argtypes = [u64, vp, u64, vp, u64]
        lib.orc_batched_coloring.restype = ctypes.c_int
        lib.orc_batched_coloring.argtypes = [u64, vp, vp, vp, vp, u64, u64, u32,
                                             vp, vp, vp, vp, vp]
        lib.orc_batched_coloring_q.restype = ctypes.c_int
        lib.orc_batched_coloring_q.argtypes = [u64, vp, vp, vp, vp, u64, u64, u32,
                                               vp, vp, vp, vp, vp, u32, ctypes.c_int]
        _LIB = lib
    return _LIB


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _csr(row_ptr, col, weight):
    rp = np.ascontiguousarray(row_ptr, dtype=np.uint64)
    cl = np.ascontiguousarray(col, dtype=np.uint32)
    wt = None if weight is None else np.ascontiguousarray(weight, dtype=np.uint32)
    return rp, cl, wt


# ---------------------------------------------------------------------------
# SplitMix64 and the per-colour weights
# ---------------------------------------------------------------------------

def mix64(z):
    return int(_lib().orc_mix64(z & (2**64 - 1)))


def splitmix_nth(state, i):
    return int(_lib().orc_splitmix_nth(state & (2**64 - 1), i))


def round_key(seed, r):
    return int(_lib().orc_round_key(seed, r))


def weight(seed, r, color, q=FP):
    """W(seed, r, b): random value of colour b in round r (Algorithm 1), in
    F_p (q = FP) or Z/2^64 (q = RING64)."""
    return int(_lib().orc_weight_q(seed, r, color, q))


def ring_preconditions(row_ptr, weight_=None):
    """Theorem 1's preconditions for Z/2^64: n <= 2^32 and every row sum
    of A at most 2^32."""
    rp = np.ascontiguousarray(row_ptr, dtype=np.uint64)
    wt = None if weight_ is None else np.ascontiguousarray(weight_, dtype=np.uint32)
    return bool(_lib().orc_ring_preconditions(rp.size - 1, _p(rp), _p(wt)))


# ---------------------------------------------------------------------------
# Oracle (a): Algorithm 1, randomized rounds
# ---------------------------------------------------------------------------

def canonicalize(labels, n=None):
    """Dense rank of each label among the distinct labels (None = all 0)."""
    if labels is None:
        out = np.zeros(n, dtype=np.uint32)
        return out, (1 if n else 0)
    lab = np.ascontiguousarray(labels, dtype=np.uint32)
    out = np.empty(lab.size, dtype=np.uint32)
    k = _lib().orc_canonicalize(lab.size, _p(lab), _p(out))
    return out, int(k)


def image(row_ptr, col, weight_, colors, k, seed, r, q=FP):
    """z = A w with w_j = W(seed, r, c_j) (Algorithm 1), mod p (q = FP) or
    mod 2^64 (q = RING64)."""
    rp, cl, wt = _csr(row_ptr, col, weight_)
    c = np.ascontiguousarray(colors, dtype=np.uint32)
    n = rp.size - 1
    z = np.empty(n, dtype=np.uint64)
    st = _lib().orc_image_q(n, _p(rp), _p(cl), _p(wt), _p(c), k, seed, r, _p(z), q)
    if st != 0:
        raise ValueError(f"orc_image_q failed ({st})")
    return z


def relabel(colors, z):
    """Rank of (c_i, z_i) among the distinct pairs, lexicographic."""
    c = np.ascontiguousarray(colors, dtype=np.uint32)
    zz = np.ascontiguousarray(z, dtype=np.uint64)
    out = np.empty(c.size, dtype=np.uint32)
    k = _lib().orc_relabel(c.size, _p(c), _p(zz), _p(out))
    return out, int(k)


def refine_round(row_ptr, col, weight_, colors, k, seed, r, q=FP):
    """One round of Algorithm 1.  Returns (new colours, k', z)."""
    rp, cl, wt = _csr(row_ptr, col, weight_)
    c = np.ascontiguousarray(colors, dtype=np.uint32)
    n = rp.size - 1
    out = np.empty(n, dtype=np.uint32)
    z = np.empty(n, dtype=np.uint64)
    k2 = _lib().orc_refine_round_q(n, _p(rp), _p(cl), _p(wt), _p(c), k, seed, r,
                                   _p(out), _p(z), q)
    if n and k2 == 0:
        raise ValueError("orc_refine_round_q: the image step failed")
    return out, int(k2), z


def stable_coloring(row_ptr, col, weight_=None, init=None, seed=0, max_rounds=0, q=FP):
    """Algorithm 1 to completion, in F_p (q = FP) or Z/2^64 (q = RING64).

    Returns (colours, k, rounds, k_per_round, status); status 0 = stable,
    1 = round cap reached, 3 = q = RING64 and Theorem 1's preconditions
    fail (nothing computed), 4 = an image step failed.
    """
    rp, cl, wt = _csr(row_ptr, col, weight_)
    n = rp.size - 1
    cap = max_rounds if max_rounds else n + 1
    lab = None if init is None else np.ascontiguousarray(init, dtype=np.uint32)
    out = np.empty(n, dtype=np.uint32)
    hist = np.zeros(max(cap, 1), dtype=np.uint32)
    k = ctypes.c_uint32(0)
    rounds = ctypes.c_uint32(0)
    st = _lib().orc_stable_coloring_q(n, _p(rp), _p(cl), _p(wt), _p(lab), seed, cap,
                                      _p(out), ctypes.byref(k), ctypes.byref(rounds),
                                      _p(hist), q)
    return out, int(k.value), int(rounds.value), hist[: rounds.value].copy(), int(st)


# ---------------------------------------------------------------------------
# Oracle (b): classic exact colour refinement and the certificate
# ---------------------------------------------------------------------------

def classic_coloring(row_ptr, col, weight_=None, init=None, max_rounds=0):
    """Classic colour refinement to its fixed point (same round convention).

    Returns (colours, k, rounds, k_per_round, status).
    """
    rp, cl, wt = _csr(row_ptr, col, weight_)
    n = rp.size - 1
    cap = max_rounds if max_rounds else n + 1
    lab = None if init is None else np.ascontiguousarray(init, dtype=np.uint32)
    out = np.empty(n, dtype=np.uint32)
    hist = np.zeros(max(cap, 1), dtype=np.uint32)
    k = ctypes.c_uint32(0)
    rounds = ctypes.c_uint32(0)
    st = _lib().orc_classic_coloring(n, _p(rp), _p(cl), _p(wt), _p(lab), cap, _p(out),
                                     ctypes.byref(k), ctypes.byref(rounds), _p(hist))
    return out, int(k.value), int(rounds.value), hist[: rounds.value].copy(), int(st)


def splitter_coloring(row_ptr, col, weight_=None, init=None):
    """Oracle (b'): the coarsest stable colouring refining ``init`` by
    splitter-based partition refinement (work list of classes, all parts
    but a largest listed on a split), the partition-refinement method of
    the baselines Section 2 discusses.  Exact and deterministic; no rounds.

    Returns (colours with first-occurrence ids, k, splitter visits), where
    the visits count the transpose entries read, O(m log n).
    Parity: pinned against brute force, automorphism orbits, closed forms
    and oracle (b) in ``tests/test_oracle_splitter.py``.
    """
    rp, cl, wt = _csr(row_ptr, col, weight_)
    n = rp.size - 1
    lab = None if init is None else np.ascontiguousarray(init, dtype=np.uint32)
    out = np.empty(n, dtype=np.uint32)
    k = ctypes.c_uint32(0)
    visits = ctypes.c_uint64(0)
    _lib().orc_splitter_coloring(n, _p(rp), _p(cl), _p(wt), _p(lab), _p(out),
                                 ctypes.byref(k), ctypes.byref(visits))
    return out, int(k.value), int(visits.value)


def classic_round(row_ptr, col, weight_, colors):
    rp, cl, wt = _csr(row_ptr, col, weight_)
    c = np.ascontiguousarray(colors, dtype=np.uint32)
    out = np.empty(c.size, dtype=np.uint32)
    k = _lib().orc_classic_round(c.size, _p(rp), _p(cl), _p(wt), _p(c), _p(out))
    return out, int(k)


def is_stable(row_ptr, col, weight_, colors):
    """Exact certificate (Definition "Stable Coloring").  Colours need not be
    dense; they are canonicalised first."""
    c, k = canonicalize(colors)
    rp, cl, wt = _csr(row_ptr, col, weight_)
    return _lib().orc_is_stable(c.size, _p(rp), _p(cl), _p(wt), _p(c), k) == 0


def first_occurrence(colors):
    c = np.ascontiguousarray(colors, dtype=np.uint32)
    out = np.empty(c.size, dtype=np.uint32)
    k = _lib().orc_first_occurrence(c.size, _p(c), _p(out))
    return out, int(k)


# ---------------------------------------------------------------------------
# Batched oracle: Algorithm 2
# ---------------------------------------------------------------------------

def batch_cut(row_ptr, max_batch):
    rp = np.ascontiguousarray(row_ptr, dtype=np.uint64)
    n = rp.size - 1
    nb = _lib().orc_batch_cut(n, _p(rp), max_batch, None, 0)
    starts = np.zeros(nb + 1, dtype=np.uint64)
    _lib().orc_batch_cut(n, _p(rp), max_batch, _p(starts), nb + 1)
    return starts


def batched_coloring(row_ptr, col, weight_=None, init=None, seed=0, max_batch=1,
                     max_rounds=0, q=FP, early_stop=False):
    """Algorithm 2 with the readings of the oracle source, in F_p (q = FP)
    or Z/2^64 (q = RING64).  early_stop adds Section 5.4's termination: the
    outer loop ends once the quotient just built would not be cut into fewer
    batches than the iteration that built it.

    Returns (first-occurrence colours, k, rounds, outer iterations,
    coarsest flag, status).
    """
    rp, cl, wt = _csr(row_ptr, col, weight_)
    n = rp.size - 1
    cap = max_rounds if max_rounds else n + 1
    lab = None if init is None else np.ascontiguousarray(init, dtype=np.uint32)
    out = np.empty(n, dtype=np.uint32)
    k = ctypes.c_uint32(0)
    rounds = ctypes.c_uint32(0)
    outer = ctypes.c_uint32(0)
    coarsest = ctypes.c_int(0)
    st = _lib().orc_batched_coloring_q(n, _p(rp), _p(cl), _p(wt), _p(lab), seed,
                                       max_batch, cap, _p(out), ctypes.byref(k),
                                       ctypes.byref(rounds), ctypes.byref(outer),
                                       ctypes.byref(coarsest), q, int(bool(early_stop)))
    return (out, int(k.value), int(rounds.value), int(outer.value),
            bool(coarsest.value), int(st))
