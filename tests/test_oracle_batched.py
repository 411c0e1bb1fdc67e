"""Pins of the batched oracle (Algorithm 2, Section 4.2).

* Theorem 2: for ANY edge partition, the merged partition of Eq. (merge) is
  stable.  Checked with random (not only contiguous) edge partitions, using
  Algorithm 1 per batch and the exact certificate.
* Batch order does not change the merged partition.
* N_b = 1 reduces to Algorithm 1 (the coarsest stable colouring).
* Termination case (i) gives the coarsest colouring; case (ii) gives a
  stable colouring that is finer than or equal to the coarsest one.
* The batch cut of the oracle: every batch <= M_b entries, batches cover the
  entry array, cuts fall on row boundaries whenever the row fits.
"""
import random

import numpy as np
import pytest

import oracle
from oracle import bruteforce as bf
from paper_2607_02603_amd import inputs


def _merged_partition(n, rp, col, batches, seed=0):
    """One outer iteration of Algorithm 2 for an arbitrary edge partition
    'batches' (list of lists of entry indices).  Returns first-occurrence
    block ids over the nodes."""
    rp = rp.astype(np.int64)
    row_of = np.repeat(np.arange(n), np.diff(rp))
    owner = {}
    for b, es in enumerate(batches):
        for e in es:
            owner.setdefault(int(row_of[e]), set()).add(b)
    key = [None] * n
    for b, es in enumerate(batches):
        inner = [i for i in range(n) if owner.get(i) == {b}]
        # restricted graph A|E_b
        es_sorted = sorted(es, key=lambda e: (row_of[e], e))
        cnt = np.zeros(n, np.int64)
        for e in es_sorted:
            cnt[row_of[e]] += 1
        brp = np.zeros(n + 1, np.uint64)
        brp[1:] = np.cumsum(cnt)
        bcol = np.array([col[e] for e in es_sorted], np.uint32)
        lab = np.zeros(n, np.uint32)
        nxt = 1
        inner_set = set(inner)
        for i in range(n):
            if i not in inner_set:
                lab[i] = nxt
                nxt += 1
        c, k, r, _, st = oracle.stable_coloring(brp, bcol, None, lab, seed=seed + b)
        assert st == 0
        for i in inner:
            key[i] = (b, int(c[i]))
    for i in range(n):
        if key[i] is None:
            key[i] = ("boundary", i)
    ids = {}
    return np.array([ids.setdefault(kk, len(ids)) for kk in key], np.uint32)


@pytest.mark.parametrize("trial", range(12))
def test_theorem2_any_edge_partition_is_stable(trial):
    rng = random.Random(300 + trial)
    n = rng.randint(5, 40)
    g = inputs.er_graph(n, rng.randint(n, 3 * n), seed=trial)
    m = g.nnz
    nb = rng.randint(2, 4)
    entries = list(range(m))
    rng.shuffle(entries)
    batches = [entries[i::nb] for i in range(nb)]
    merged = _merged_partition(n, g.row_ptr, g.col, batches)
    assert oracle.is_stable(g.row_ptr, g.col, None, merged)
    # finer than or equal to the coarsest stable colouring
    S = oracle.first_occurrence(oracle.stable_coloring(g.row_ptr, g.col)[0])[0]
    for blk in set(merged.tolist()):
        assert len(set(S[merged == blk].tolist())) == 1
    # batch order does not matter (merge = meet on the partition lattice)
    shuffled = list(reversed(batches))
    merged2 = _merged_partition(n, g.row_ptr, g.col, shuffled, seed=77)
    assert bf.partition_of(merged2) == bf.partition_of(merged)


@pytest.mark.parametrize("mb", [1, 3, 8, 50, 10**9])
def test_batch_cut(mb):
    g = inputs.rmat(8, 4, seed=2)
    starts = oracle.batch_cut(g.row_ptr, mb).astype(np.int64)
    m = g.nnz
    assert starts[0] == 0 and starts[-1] == m
    sizes = np.diff(starts)
    assert np.all(sizes <= mb) and np.all(sizes >= 0)
    if m > 0:
        assert np.all(sizes > 0)
    rp = set(g.row_ptr.astype(np.int64).tolist())
    deg = np.diff(g.row_ptr.astype(np.int64))
    # a cut inside a row only when that row does not fit in one batch
    for s in starts[1:-1]:
        if s not in rp:
            row = np.searchsorted(g.row_ptr.astype(np.int64), s, side="right") - 1
            assert deg[row] > 0
    if mb >= m:
        assert len(starts) == 2


def test_single_batch_equals_in_core():
    g = inputs.rmat(10, 8, seed=5)
    c, k, r, outer, coarsest, st = oracle.batched_coloring(g.row_ptr, g.col,
                                                           max_batch=10**9)
    ref, kr, rr, _, _ = oracle.stable_coloring(g.row_ptr, g.col)
    assert st == 0 and coarsest and outer == 1
    assert np.array_equal(c, oracle.first_occurrence(ref)[0])
    assert k == kr and r == rr


@pytest.mark.parametrize("mb", [8, 40, 200, 1000])
def test_batched_stable_and_case_i_is_coarsest(mb):
    g = inputs.rmat(9, 6, seed=6)
    c, k, r, outer, coarsest, st = oracle.batched_coloring(g.row_ptr, g.col,
                                                           max_batch=mb)
    assert st == 0
    assert oracle.is_stable(g.row_ptr, g.col, None, c)
    S = oracle.first_occurrence(oracle.stable_coloring(g.row_ptr, g.col)[0])[0]
    for blk in range(k):
        assert len(set(S[c == blk].tolist())) == 1
    if coarsest:
        assert np.array_equal(c, S)
    assert outer >= 1


def test_tiny_cap_forces_several_outer_iterations():
    # 30 disjoint paths P4: batches hold whole paths, so every batch merges
    # and the quotient shrinks; contraction ends with one batch (case (i)).
    edges = [(4 * t + i, 4 * t + i + 1) for t in range(30) for i in range(3)]
    rp, col = bf.to_csr(120, edges)
    c, k, r, outer, coarsest, st = oracle.batched_coloring(rp, col, max_batch=12)
    assert outer >= 2 and coarsest and k == 2
    assert oracle.is_stable(rp, col, None, c)
    # a grid with the same cap does not contract at all: case (ii) at once
    g = inputs.grid_graph(6, 7)
    c, k, r, outer, coarsest, st = oracle.batched_coloring(g.row_ptr, g.col,
                                                           max_batch=12)
    assert outer == 1 and not coarsest and k == g.n
    assert oracle.is_stable(g.row_ptr, g.col, None, c)


def test_batched_respects_initial_partition():
    rp, col = bf.to_csr(8, [(i, (i + 1) % 8) for i in range(8)])
    init = np.array([0, 0, 0, 1, 0, 0, 0, 0], np.uint32)
    c, *_ = oracle.batched_coloring(rp, col, init=init, max_batch=5)
    assert c[3] != c[2] and c[3] != c[4]
    assert oracle.is_stable(rp, col, None, c)


def test_batched_weighted_quotient_input():
    # weighted directed input: quotients of quotients stay consistent
    rng = random.Random(4)
    n = 30
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(120)]
    rp, col = bf.to_csr(n, edges, directed=True)
    wt = np.array([rng.randint(1, 3) for _ in range(col.size)], np.uint32)
    for mb in (7, 25, 1000):
        c, k, r, outer, coarsest, st = oracle.batched_coloring(rp, col, wt, max_batch=mb)
        assert st == 0
        assert oracle.is_stable(rp, col, wt, c)
        truth = bf.partition_of(oracle.stable_coloring(rp, col, wt)[0])
        if coarsest:
            assert bf.partition_of(c) == truth


def _path_with_isolated(L, every):
    """Path 0-1-...-(L-1) on the path nodes, with an isolated node inserted
    after every 'every' path nodes.  Returns (rp, col, is_path)."""
    order = []
    p = 0
    while p < L:
        for _ in range(min(every, L - p)):
            order.append(("p", p))
            p += 1
        order.append(("iso", None))
    n = len(order)
    node_of_path = {}
    for v, (kind, idx) in enumerate(order):
        if kind == "p":
            node_of_path[idx] = v
    edges = [(node_of_path[i], node_of_path[i + 1]) for i in range(L - 1)]
    rp, col = bf.to_csr(n, edges)
    is_path = np.array([kind == "p" for kind, _ in order])
    return rp, col, is_path


@pytest.mark.parametrize("L,every,mb", [(60, 5, 14), (200, 7, 31), (90, 3, 20)])
def test_early_stop_fires_after_first_iteration(L, every, mb):
    """Section 5.4's termination on a path with isolated nodes spread over
    it.  Rows never exceed the cap, so every node is inner to the batch that
    holds its row.  Within a batch, the path nodes are pinned by the frozen
    singletons next to the batch (or by the path's end) and all end up as
    singletons; the isolated nodes of a batch share z = 0 in every round and
    form one block.  The quotient therefore keeps every entry, is cut into
    the same ranges, and the early stop ends the loop after one outer
    iteration.  Without it, the second iteration merges nothing more (each
    batch now holds a single isolated block) and ends at the fixed point."""
    rp, col, is_path = _path_with_isolated(L, every)
    n = rp.size - 1
    starts = oracle.batch_cut(rp, mb).astype(np.int64)
    nb = starts.size - 1
    assert nb >= 2
    # batch of every isolated row: the range that holds its start offset
    iso = np.flatnonzero(~is_path)
    off = rp.astype(np.int64)[iso]
    bat = np.minimum(np.searchsorted(starts, off, side="right") - 1, nb - 1)
    want_k = L + len(set(bat.tolist()))
    # expected colouring: path nodes singletons, one block per batch of
    # isolated rows, numbered by first occurrence
    key = [("p", v) if is_path[v] else ("b", int(bat[np.searchsorted(iso, v)]))
           for v in range(n)]
    ids = {}
    want = np.array([ids.setdefault(kk, len(ids)) for kk in key], np.uint32)

    c, k, r, outer, coarsest, st = oracle.batched_coloring(rp, col, max_batch=mb,
                                                           early_stop=True)
    assert st == 0 and outer == 1 and not coarsest
    assert k == want_k and np.array_equal(c, want)
    c2, k2, r2, outer2, coarsest2, st2 = oracle.batched_coloring(rp, col, max_batch=mb)
    assert st2 == 0 and outer2 == 2 and not coarsest2
    assert np.array_equal(c2, c) and r2 > r
    assert oracle.is_stable(rp, col, None, c)


def test_early_stop_does_not_fire_while_batches_shrink():
    # 30 disjoint P4s, two per batch: every batch contracts to 2 blocks and
    # 3 entries, so each quotient needs fewer batches and the loop runs on
    # to a single batch (case (i)), exactly as without the early stop
    edges = [(4 * t + i, 4 * t + i + 1) for t in range(30) for i in range(3)]
    rp, col = bf.to_csr(120, edges)
    plain = oracle.batched_coloring(rp, col, max_batch=12)
    early = oracle.batched_coloring(rp, col, max_batch=12, early_stop=True)
    assert plain[4] and early[4] and plain[3] >= 2
    assert np.array_equal(plain[0], early[0]) and plain[1:5] == early[1:5]


@pytest.mark.parametrize("seed,mb", [(1, 40), (2, 120), (3, 300), (4, 900)])
def test_early_stop_is_a_prefix_of_the_plain_loop(seed, mb):
    """The early stop only ends the outer loop sooner: it runs the same
    iterations as the plain loop up to that point, so its colouring is
    stable (Theorem 2), is refined into by nothing the plain loop does
    differently (the plain colouring is a coarsening of it), and equals the
    plain one whenever both ran the same number of outer iterations."""
    g = inputs.rmat(9, 8, seed=seed)
    c, k, r, outer, coarsest, st = oracle.batched_coloring(g.row_ptr, g.col, max_batch=mb,
                                                           early_stop=True)
    cp, kp, rp_, outerp, coarsestp, stp = oracle.batched_coloring(g.row_ptr, g.col,
                                                                  max_batch=mb)
    assert st == 0 and stp == 0
    assert 1 <= outer <= outerp and r <= rp_ and k >= kp
    assert oracle.is_stable(g.row_ptr, g.col, None, c)
    for blk in range(k):
        assert len(set(cp[c == blk].tolist())) == 1
    if outer == outerp:
        assert np.array_equal(c, cp) and coarsest == coarsestp
    if coarsest:
        assert outer == outerp
