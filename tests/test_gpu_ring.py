"""GPU parity in the ring Z/2^64 (Algorithm 1 with precision q = 64,
Section 4.1): the HIP path, switched with wl_set_precision, against the
oracle in the same arithmetic.  Bit-exact colour ids, colour count and round
count for Algorithm 1 (in core, propagation blocking, device-driven rounds,
single rounds, streamed), first-occurrence colours for Algorithm 2; the
partition equals the one of F_p mode and of classic refinement.  Theorem 1's
row-sum bound is enforced on every path.
"""
import random

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02603_amd as wl
from oracle import bruteforce as bf
from paper_2607_02603_amd import inputs

import ring_cases

pytestmark = pytest.mark.gpu
R = oracle.RING64


@pytest.fixture(autouse=True)
def ring():
    prev = wl.wl_get_precision()
    wl.wl_set_precision(wl.WL_PRECISION_RING64)
    yield
    wl.wl_set_precision(prev)


def _say(msg):
    print(msg, flush=True)


def _init_t(init, device="cuda"):
    if init is None:
        return None
    t = torch.from_numpy(np.asarray(init, np.uint32).view(np.int32))
    return t.cuda() if device == "cuda" else t


def _dev_graph(rp, col, wt=None, rp64=False, symmetric=False):
    n = len(rp) - 1
    rp = np.asarray(rp, np.uint64)
    if not rp64:
        rp = rp.astype(np.uint32)
    return wl.Graph.from_numpy(n, rp, col, wt, device="cuda", symmetric=symmetric)


def _exact(rp, col, wt=None, init=None, seed=0, rp64=False, symmetric=False, classic=True):
    g = _dev_graph(rp, col, wt, rp64, symmetric)
    c, k, r = wl.wl_stable_coloring(g, _init_t(init), seed)
    got = c.cpu().numpy().view(np.uint32)
    co, ko, ro, _, st = oracle.stable_coloring(rp, col, wt, init, seed, q=R)
    assert st == 0
    assert (k, r) == (ko, ro)
    assert np.array_equal(got, co)
    if classic:
        cb = oracle.classic_coloring(rp, col, wt, init)[0]
        assert np.array_equal(oracle.first_occurrence(got)[0], oracle.first_occurrence(cb)[0])
    return got, k, r


@pytest.mark.parametrize("trial", range(16))
def test_random_small_graphs(trial):
    rng = random.Random(300 + trial)
    n = rng.randint(1, 300)
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(0, 4 * n))]
    rp, col = bf.to_csr(n, edges, directed=trial % 2 == 1)
    wt = None
    if trial % 3 == 2:
        # large weights: products and sums wrap past 2^64 (row sums <= 2^32)
        wt = np.array([rng.choice([1, 2, 3, 1 << 28, (1 << 31) - 1]) for _ in range(col.size)],
                      np.uint32)
        if not oracle.ring_preconditions(rp, wt):
            wt = (wt & 0xFFFFF).astype(np.uint32) | 1
    init = None
    if trial % 4 == 3:
        init = np.array([rng.choice([7, 100, 2**31 + 5]) for _ in range(n)], np.uint32)
    _say(f"ring random trial={trial} n={n} nnz={col.size}")
    _exact(rp, col, wt, init, seed=trial)


def test_path_grid_and_edgeless():
    for n in (1, 2, 5, 12, 101):
        rp, col = bf.to_csr(n, [(i, i + 1) for i in range(n - 1)])
        _, k, r = _exact(rp, col)
        assert k == (n + 1) // 2
    g = inputs.grid_graph(40)
    _, k, r = _exact(g.row_ptr, g.col)
    assert (k, r) == (210, 20)


def test_heavy_rows_and_large_classes():
    rng = random.Random(11)
    edges = [(0, i) for i in range(1, 10001)]
    n = 10001
    hubs = []
    for h in range(40):
        hub = n
        n += 1
        hubs.append(hub)
        for _ in range(h * 50 + 3):
            edges.append((hub, n))
            n += 1
    for _ in range(3000):
        prev = rng.choice(hubs)
        for _ in range(rng.randint(1, 4)):
            edges.append((prev, n))
            prev = n
            n += 1
    rp, col = bf.to_csr(n, edges)
    _say(f"ring heavy n={n}")
    _exact(rp, col, seed=3)
    _exact(rp, col, seed=4, rp64=True)
    # a weighted heavy row (10000 entries of weight 2^18, row sum < 2^32)
    wt = np.ones(col.size, np.uint32)
    wt[: 10000] = 1 << 18
    assert oracle.ring_preconditions(rp, wt)
    _exact(rp, col, wt, seed=6)


def test_radix_passes_many_distinct_in_one_class():
    edges = []
    n = 0
    for h in range(200):
        hub = n
        n += 1
        for _ in range(h + 1):
            edges.append((hub, n))
            n += 1
    rp, col = bf.to_csr(n, edges)
    _exact(rp, col, seed=5)


def test_largest_key_in_every_sort():
    # z = 2^64 - 1 (the padding key of the sorting networks) on members of
    # classes of 6, 50, 1000 and 5000 nodes: the pico, tiny, LDS and radix
    # sorts of round 0 must keep every member and drop every padding slot
    rp, col, wt, lab, seed, tn = ring_cases.max_key_graph()
    c0, k0 = oracle.canonicalize(lab)
    z = oracle.image(rp, col, wt, c0, k0, seed, 0, R)
    assert sorted(np.nonzero(z == np.uint64(2**64 - 1))[0].tolist()) == tn
    _say(f"ring max key seed={seed} targets={len(tn)}")
    _exact(rp, col, wt, lab, seed=seed, classic=False)
    g = _dev_graph(rp, col, wt)
    cin = torch.from_numpy(c0.view(np.int32)).cuda()
    cout, kg = wl.wl_refine_round(g, cin, k0, seed, 0)
    c1, k1, _ = oracle.refine_round(rp, col, wt, c0, k0, seed, 0, q=R)
    assert kg == k1 and np.array_equal(cout.cpu().numpy().view(np.uint32), c1)


def test_many_colours_full_table_mode():
    # more than 65535 colours: each value computed from the neighbour's colour
    g = inputs.er_graph(100000, 400000, seed=2)
    _say(f"ring er100k nnz={g.nnz}")
    _, k, _ = _exact(g.row_ptr, g.col, seed=1, classic=False)
    assert k > 65535


def test_weighted_quotient_like_graph():
    rng = random.Random(8)
    n = 3000
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(20000)]
    rp, col = bf.to_csr(n, edges, directed=True)
    wt = np.array([rng.randint(1, 2**28) for _ in range(col.size)], np.uint32)
    assert oracle.ring_preconditions(rp, wt)
    _exact(rp, col, wt, seed=9)


def test_partition_equals_fp_mode():
    g = inputs.rmat(14, 8, seed=4)
    got, k, r = _exact(g.row_ptr, g.col, seed=2, classic=False)
    dg = _dev_graph(g.row_ptr, g.col)
    with wl.precision(wl.WL_PRECISION_FP):
        cf, kf, rf = wl.wl_stable_coloring(dg, None, 2)
    assert (kf, rf) == (k, r)
    assert np.array_equal(oracle.first_occurrence(got)[0],
                          oracle.first_occurrence(cf.cpu().numpy().view(np.uint32))[0])


def test_refine_round_each_round():
    g = inputs.rmat(13, 8, seed=1)
    dg = _dev_graph(g.row_ptr, g.col)
    c, k = oracle.canonicalize(None, g.n)
    r = 0
    while True:
        cin = torch.from_numpy(c.view(np.int32)).cuda()
        cout, kg = wl.wl_refine_round(dg, cin, k, 17, r)
        c2, k2, _ = oracle.refine_round(g.row_ptr, g.col, None, c, k, 17, r, q=R)
        assert kg == k2
        assert np.array_equal(cout.cpu().numpy().view(np.uint32), c2)
        r += 1
        if k2 == k:
            break
        c, k = c2, k2
    assert r >= 3


# ---------------------------------------------------------------------------
# propagation blocking (symmetric unweighted graphs)
# ---------------------------------------------------------------------------

def test_propagation_blocking(monkeypatch):
    monkeypatch.setenv("WL_PB", "force")
    rng = random.Random(5)
    for trial in range(4):
        n = rng.randint(50, 5000)
        edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(n, 6 * n))]
        edges = [(u, v) for u, v in edges if u != v]
        rp, col = bf.to_csr(n, edges)
        _exact(rp, col, seed=trial, symmetric=True)
    # a star: one bin of many slices, whole waves feeding one row
    rp, col = bf.to_csr(70001, [(0, i) for i in range(1, 70001)])
    _exact(rp, col, seed=7, symmetric=True)
    g = inputs.rmat(14, 8, seed=3)
    _exact(g.row_ptr, g.col, seed=3, symmetric=True, classic=False)


# ---------------------------------------------------------------------------
# device-driven rounds
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("host_rounds,passes,graph", [(0, 0, 0), (0, 2, 0), (3, 1, 0),
                                                      (0, 1, 1)])
def test_device_driven_rounds(monkeypatch, host_rounds, passes, graph):
    monkeypatch.setenv("WL_HOST_ROUNDS", str(host_rounds))
    monkeypatch.setenv("WL_ASYNC_PASSES", str(passes))
    monkeypatch.setenv("WL_GRAPH", str(graph))
    g = inputs.grid_graph(64)
    _exact(g.row_ptr, g.col, seed=1, classic=False)
    rp, col, wt, lab, seed, _ = ring_cases.max_key_graph()
    _exact(rp, col, wt, lab, seed=seed, classic=False)


# ---------------------------------------------------------------------------
# host-memory paths
# ---------------------------------------------------------------------------

def _host_graph(rp, col, wt=None, pinned=True):
    n = len(rp) - 1
    g = wl.Graph.from_numpy(n, np.asarray(rp, np.uint64), col, wt, device=None)
    if not pinned:
        return g
    return wl.Graph(n, g.row_ptr.pin_memory(), g.col_idx.pin_memory(),
                    None if g.weight is None else g.weight.pin_memory())


def _ws_for_chunk(n, entries, weighted):
    import ctypes
    s = wl.WlCsr()
    s.n = n
    s.nnz = entries
    s.weight = 8 if weighted else None
    out = ctypes.c_uint64(0)
    assert wl.lib().wl_streamed_workspace_size(ctypes.byref(s), ctypes.byref(out)) == 0
    return int(out.value)


@pytest.mark.parametrize("chunk", [None, 5000])
def test_streamed(chunk):
    rng = random.Random(21)
    n = 3000
    edges = [(0, 1 + rng.randrange(n - 1)) for _ in range(15000)]
    edges += [(rng.randrange(n), rng.randrange(n)) for _ in range(12000)]
    rp, col = bf.to_csr(n, edges, directed=True)
    wt = np.array([rng.randint(1, 1 << 17) for _ in range(col.size)], np.uint32)
    for w in (None, wt):
        g = _host_graph(rp, col, w)
        ws = None if chunk is None else _ws_for_chunk(n, chunk, w is not None)
        c, k, r = wl.wl_stable_coloring_streamed(g, None, 4, ws_bytes=ws)
        co, ko, ro, _, st = oracle.stable_coloring(rp, col, w, None, 4, q=R)
        assert st == 0 and (k, r) == (ko, ro)
        assert np.array_equal(c.numpy().view(np.uint32), co)
    rp, col, wt, lab, seed, _ = ring_cases.max_key_graph()
    c, k, r = wl.wl_stable_coloring_streamed(_host_graph(rp, col, wt), _init_t(lab, "cpu"), seed)
    co, ko, ro, _, st = oracle.stable_coloring(rp, col, wt, lab, seed, q=R)
    assert (k, r) == (ko, ro) and np.array_equal(c.numpy().view(np.uint32), co)


@pytest.mark.parametrize("mb", [3, 40, 10**9])
def test_batched(mb):
    g = inputs.rmat(10, 6, seed=6)
    hg = _host_graph(g.row_ptr, g.col)
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(hg, None, 0, mb)
    ref, kr, rr, orr, cr, st = oracle.batched_coloring(g.row_ptr, g.col, None, None, 0, mb,
                                                       q=R)
    got = c.numpy().view(np.uint32)
    assert st == 0
    assert np.array_equal(got, ref)
    assert (k, outer, coarsest, r) == (kr, orr, cr, rr)
    c2, *_ = wl.wl_stable_coloring_batched(hg, None, 0, mb, options=wl.WL_BATCHED_EXACT)
    coarsest_ref = oracle.first_occurrence(oracle.classic_coloring(g.row_ptr, g.col)[0])[0]
    assert np.array_equal(c2.numpy().view(np.uint32), coarsest_ref)


def test_batched_weighted_directed():
    rng = random.Random(77)
    n = 250
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(1200)]
    rp, col = bf.to_csr(n, edges, directed=True)
    wt = np.array([rng.randint(1, 1 << 20) for _ in range(col.size)], np.uint32)
    init = np.array([rng.choice([3, 9]) for _ in range(n)], np.uint32)
    g = _host_graph(rp, col, wt)
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(g, _init_t(init, "cpu"), 0, 17)
    ref, kr, rr, orr, cr, st = oracle.batched_coloring(rp, col, wt, init, 0, 17, q=R)
    assert st == 0 and np.array_equal(c.numpy().view(np.uint32), ref)
    assert (k, outer, coarsest, r) == (kr, orr, cr, rr)


# ---------------------------------------------------------------------------
# Theorem 1's bound on the row sums
# ---------------------------------------------------------------------------

def test_row_sum_bound_every_path():
    rp = np.array([0, 3, 3, 4], np.uint64)
    col = np.array([1, 1, 2, 0], np.uint32)
    ok = np.array([1 << 31, (1 << 31) - 1, 1, 5], np.uint32)   # row sum 2^32
    bad = np.array([1 << 31, (1 << 31) - 1, 2, 5], np.uint32)  # 2^32 + 1
    _exact(rp, col, ok, classic=False)
    with pytest.raises(wl.WlError) as e:
        wl.wl_stable_coloring(_dev_graph(rp, col, bad), None, 0)
    assert e.value.code == wl.WL_EOVERFLOW
    cin = torch.zeros(3, dtype=torch.int32, device="cuda")
    with pytest.raises(wl.WlError) as e:
        wl.wl_refine_round(_dev_graph(rp, col, bad), cin, 1, 0, 0)
    assert e.value.code == wl.WL_EOVERFLOW
    with pytest.raises(wl.WlError) as e:
        wl.wl_stable_coloring_streamed(_host_graph(rp, col, bad), None, 0)
    assert e.value.code == wl.WL_EOVERFLOW
    with pytest.raises(wl.WlError) as e:
        wl.wl_stable_coloring_batched(_host_graph(rp, col, bad), None, 0, 2)
    assert e.value.code == wl.WL_EOVERFLOW
    # a row of 100 weights (summed by a whole wave) at and above the bound
    n = 101
    rp = np.array([0, 100] + [100] * (n - 1), np.uint64)
    col = np.arange(1, 101, dtype=np.uint32)
    wide = np.full(100, 1 << 25, np.uint32)
    wide[0] = (1 << 32) - 99 * (1 << 25)
    assert int(wide.astype(np.uint64).sum()) == 1 << 32
    _exact(rp, col, wide, classic=False)
    wide[1] += 1
    with pytest.raises(wl.WlError) as e:
        wl.wl_stable_coloring(_dev_graph(rp, col, wide), None, 0)
    assert e.value.code == wl.WL_EOVERFLOW
    # F_p has no such bound
    with wl.precision(wl.WL_PRECISION_FP):
        c, k, r = wl.wl_stable_coloring(_dev_graph(rp, col, bad), None, 0)
    co, ko, ro, _, _ = oracle.stable_coloring(rp, col, bad, None, 0)
    assert (k, r) == (ko, ro) and np.array_equal(c.cpu().numpy().view(np.uint32), co)
