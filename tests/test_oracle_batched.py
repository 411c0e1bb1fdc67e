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
