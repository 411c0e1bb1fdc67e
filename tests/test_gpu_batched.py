"""GPU parity of Algorithm 2 (wl_stable_coloring_batched) with the batched
oracle: identical first-occurrence colours, colour count, rounds summed over
the batch runs, outer iterations and the coarsest flag."""
import random

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02603_amd as wl
from oracle import bruteforce as bf
from paper_2607_02603_amd import inputs

pytestmark = pytest.mark.gpu


def _host_graph(rp, col, wt=None, pinned=True):
    n = len(rp) - 1
    g = wl.Graph.from_numpy(n, rp, col, wt, device=None)
    if not pinned:
        return g
    return wl.Graph(n, g.row_ptr.pin_memory(), g.col_idx.pin_memory(),
                    None if g.weight is None else g.weight.pin_memory())


def _check(rp, col, wt=None, init=None, mb=8, seed=0, pinned=True, early=False):
    g = _host_graph(rp, col, wt, pinned)
    init_t = None if init is None else torch.from_numpy(np.asarray(init, np.uint32).view(np.int32))
    opts = wl.WL_BATCHED_EARLY_STOP if early else 0
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(g, init_t, seed, mb, options=opts)
    got = c.numpy().view(np.uint32)
    ref, kr, rr, orr, cr, st = oracle.batched_coloring(rp, col, wt, init, seed, mb,
                                                       early_stop=early)
    assert st == 0
    assert np.array_equal(got, ref)
    assert (k, outer, coarsest) == (kr, orr, cr)
    assert r == rr
    assert oracle.is_stable(rp, col, wt, got)
    return got, k, r, outer, coarsest


@pytest.mark.parametrize("mb", [1, 3, 8, 40, 300, 10**9])
def test_rmat_small_various_caps(mb):
    g = inputs.rmat(9, 6, seed=6)
    print(f"rmat9 mb={mb}", flush=True)
    _check(g.row_ptr, g.col, mb=mb, seed=mb)


def test_single_batch_equals_in_core():
    g = inputs.rmat(11, 8, seed=5)
    got, k, r, outer, coarsest = _check(g.row_ptr, g.col, mb=10**9)
    assert coarsest and outer == 1
    ref = oracle.stable_coloring(g.row_ptr, g.col)[0]
    assert np.array_equal(got, oracle.first_occurrence(ref)[0])


def test_disjoint_paths_contract_to_coarsest():
    edges = [(4 * t + i, 4 * t + i + 1) for t in range(30) for i in range(3)]
    rp, col = bf.to_csr(120, edges)
    got, k, r, outer, coarsest = _check(rp, col, mb=12)
    assert outer >= 2 and coarsest and k == 2


def test_grid_fixed_point_case_ii():
    g = inputs.grid_graph(6, 7)
    got, k, r, outer, coarsest = _check(g.row_ptr, g.col, mb=12)
    assert outer == 1 and not coarsest


@pytest.mark.parametrize("trial", range(6))
def test_random_weighted_directed(trial):
    rng = random.Random(40 + trial)
    n = rng.randint(5, 200)
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(n, 6 * n))]
    rp, col = bf.to_csr(n, edges, directed=True)
    wt = np.array([rng.randint(1, 5) for _ in range(col.size)], np.uint32)
    init = None
    if trial % 2:
        init = np.array([rng.choice([3, 9]) for _ in range(n)], np.uint32)
    for mb in (5, 37, 10**6):
        _check(rp, col, wt, init, mb=mb, seed=trial)


def test_long_multi_edge_row_quotient_pieces():
    # a row with far more entries than nodes: the quotient phase cuts it
    # into pieces when the workspace is tight
    n = 12
    edges = [(0, 1 + (i % 11)) for i in range(3000)] + [(i, i + 1) for i in range(1, 11)]
    rp, col = bf.to_csr(n, edges, directed=True)
    g = _host_graph(rp, col)
    mb = 16
    need = wl.wl_batched_workspace_size(g, mb)
    ws = wl.workspace(need)
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(g, None, 0, mb, ws=ws)
    ref, kr, rr, orr, cr, st = oracle.batched_coloring(rp, col, None, None, 0, mb)
    assert np.array_equal(c.numpy().view(np.uint32), ref)
    assert (k, r, outer, coarsest) == (kr, rr, orr, cr)


def test_edge_cases():
    # edgeless graph, one node, empty graph
    for n in (1, 5):
        rp = np.zeros(n + 1, np.uint64)
        col = np.zeros(0, np.uint32)
        _check(rp, col, mb=4)
    g = _host_graph(np.zeros(1, np.uint64), np.zeros(0, np.uint32))
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(g, None, 0, 4)
    assert (k, r) == (0, 0)


def test_budget_errors():
    g0 = inputs.rmat(8, 4, seed=1)
    g = _host_graph(g0.row_ptr, g0.col)
    need = wl.wl_batched_workspace_size(g, 50)
    ws = wl.workspace(need)
    # a larger cap than the workspace allows
    with pytest.raises(wl.WlError) as e:
        wl.wl_stable_coloring_batched(g, None, 0, 10**9, ws=ws)
    assert e.value.code == wl.WL_EBUDGET
    # cap 0 = the largest that fits: still a valid, stable result
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(g, None, 0, 0, ws=ws)
    assert oracle.is_stable(g0.row_ptr, g0.col, None, c.numpy().view(np.uint32))


def test_medium_rmat_explicit_cap():
    g = inputs.rmat(18, 16, seed=3)
    print("rmat18 explicit cap", flush=True)
    got, k, r, outer, coarsest = _check(g.row_ptr, g.col, mb=g.nnz // 6)


@pytest.mark.parametrize("mb", [5, 64, 10**9])
def test_pageable_host_graph(mb):
    # the same graphs from pageable host memory (copied through the library's
    # page-locked staging buffers) give the oracle's result
    g = inputs.rmat(9, 8, seed=1)
    _check(g.row_ptr, g.col, mb=mb, pinned=False)
    rng = random.Random(mb)
    n = 300
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(2000)]
    rp, col = bf.to_csr(n, edges, directed=True)
    wt = np.array([rng.randint(1, 4) for _ in range(col.size)], np.uint32)
    _check(rp, col, wt, mb=mb, pinned=False)


def test_medium_rmat_pageable_explicit_cap():
    # several outer iterations with quotients larger than one staging buffer
    g = inputs.rmat(18, 16, seed=5)
    print("rmat18 pageable explicit cap", flush=True)
    _check(g.row_ptr, g.col, mb=g.nnz // 5, pinned=False)


def test_medium_rmat_tight_budget_auto_cap():
    # R-MAT scale 18 in pinned host memory with a workspace far smaller than
    # one in-core run needs: several batches, cap chosen by the library.
    g0 = inputs.rmat(18, 16, seed=3)
    g = _host_graph(g0.row_ptr, g0.col)
    ws = wl.workspace(wl.wl_batched_workspace_size(g, g.nnz // 6))
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(g, None, 0, 0, ws=ws)
    got = c.numpy().view(np.uint32)
    print(f"rmat18 auto cap: k={k} rounds={r} outer={outer} coarsest={coarsest}", flush=True)
    assert oracle.is_stable(g0.row_ptr, g0.col, None, got)
    ref = oracle.first_occurrence(oracle.stable_coloring(g0.row_ptr, g0.col)[0])[0]
    S = ref
    for blk in np.unique(got)[:2000]:
        assert len(np.unique(S[got == blk])) == 1  # finer than or equal to coarsest
    if coarsest:
        assert np.array_equal(got, ref)


def test_rmat20_several_outer_iterations():
    # R-MAT scale 20 (31M entries) under a cap of a fifth of the entries:
    # several batches with heavy rows and several outer iterations; the same
    # result twice
    g = inputs.rmat(20, 16, seed=3)
    mb = g.nnz // 5
    print(f"rmat20 mb={mb}", flush=True)
    got, k, r, outer, coarsest = _check(g.row_ptr, g.col, mb=mb)
    assert outer >= 2
    again = wl.wl_stable_coloring_batched(_host_graph(g.row_ptr, g.col), None, 0, mb)
    assert np.array_equal(again[0].numpy().view(np.uint32), got)
    # with the exact finish, after the fixed point or the early stop: the
    # coarsest colouring (the quotient pipeline's chunks, then the streamed
    # rounds on a weighted quotient)
    ref = oracle.first_occurrence(oracle.stable_coloring(g.row_ptr, g.col, None, None, 0)[0])[0]
    for opt in (wl.WL_BATCHED_EXACT, wl.WL_BATCHED_EXACT | wl.WL_BATCHED_EARLY_STOP):
        c, k2, r2, outer2, co = wl.wl_stable_coloring_batched(_host_graph(g.row_ptr, g.col),
                                                              None, 0, mb, options=opt)
        print(f"rmat20 options={opt}: outer={outer2} colours={k2}", flush=True)
        assert co and np.array_equal(c.numpy().view(np.uint32), ref)


def test_pageable_copies_without_staging(monkeypatch):
    # the copies from and to pageable memory as they run when page-locked
    # staging is refused (Algorithm 2's batches and quotients, the exact
    # finish and the streamed rounds)
    monkeypatch.setenv("WL_HOST_STAGING", "0")
    g = inputs.rmat(12, 8, seed=5)
    for mb in (3000, 40000):
        _check(g.row_ptr, g.col, mb=mb, seed=2, pinned=False)
    hg = _host_graph(g.row_ptr, g.col, pinned=False)
    c, k, r, outer, coarsest = wl.wl_stable_coloring_batched(hg, None, 0, 5000,
                                                             options=wl.WL_BATCHED_EXACT)
    ref = oracle.first_occurrence(oracle.stable_coloring(g.row_ptr, g.col, None, None, 0)[0])[0]
    assert coarsest and np.array_equal(c.numpy().view(np.uint32), ref)
    c, k, r = wl.wl_stable_coloring_streamed(hg, None, 3)
    co, ko, ro, _, _ = oracle.stable_coloring(g.row_ptr, g.col, None, None, 3)
    assert (k, r) == (ko, ro) and np.array_equal(c.numpy().view(np.uint32), co)


# Section 5.4's early stop (WL_BATCHED_EARLY_STOP without the exact finish)
# against the batched oracle with the same rule: colours, colour count,
# rounds, outer iterations and the coarsest flag.

@pytest.mark.parametrize("seed,mb", [(1, 40), (2, 120), (3, 300), (4, 900), (6, 3)])
def test_early_stop_rmat(seed, mb):
    g = inputs.rmat(9, 8, seed=seed)
    print(f"early stop rmat9 seed={seed} mb={mb}", flush=True)
    _check(g.row_ptr, g.col, mb=mb, seed=seed, early=True)


def test_early_stop_path_with_isolated_nodes():
    # the rule fires after the first outer iteration (the quotient keeps
    # every entry); the oracle's pins derive that in closed form
    L, every, mb = 200, 7, 31
    order = []
    p = 0
    while p < L:
        for _ in range(min(every, L - p)):
            order.append(p)
            p += 1
        order.append(-1)
    node = {v: i for i, v in enumerate(order) if v >= 0}
    rp, col = bf.to_csr(len(order), [(node[i], node[i + 1]) for i in range(L - 1)])
    got, k, r, outer, coarsest = _check(rp, col, mb=mb, early=True)
    assert outer == 1 and not coarsest


@pytest.mark.parametrize("trial", range(4))
def test_early_stop_weighted_labels(trial):
    rng = random.Random(90 + trial)
    n = rng.randint(50, 400)
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(n, 6 * n))]
    rp, col = bf.to_csr(n, edges, directed=True)
    wt = np.array([rng.randint(1, 5) for _ in range(col.size)], np.uint32)
    init = np.array([rng.choice([3, 9]) for _ in range(n)], np.uint32) if trial % 2 else None
    for mb in (9, 60, 10**6):
        _check(rp, col, wt, init, mb=mb, seed=trial, pinned=bool(trial % 2), early=True)


def test_early_stop_rmat_larger():
    # R-MAT scale 14: several batches and outer iterations
    g = inputs.rmat(14, 8, seed=3)
    for mb in (20000, 60000):
        print(f"early stop rmat14 mb={mb}", flush=True)
        _check(g.row_ptr, g.col, mb=mb, seed=5, early=True)
