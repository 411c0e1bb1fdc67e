"""Pins of the oracle's ring arithmetic (Algorithm 1 with precision q = 64:
values, sums and products in Z/2^64, Section 4.1) against things other than
itself.

* The ring values are the unreduced SplitMix64 outputs whose residues mod p
  are the F_p values (pinned by the published outputs in
  test_oracle_pins.py), spread over all of [0, 2^64), pairwise distinct.
* Closed forms of the image: products with powers of two shift the value
  (bits above 2^64 drop out), long rows of the largest weights wrap.
* Linearity of A -> A w over Z/2^64.
* Partitions: exhaustive search on tiny graphs, closed forms and symmetry
  orbits, classic refinement on larger random graphs (Theorem 1 makes the
  ring result the coarsest stable colouring, as in F_p).
* Theorem 1's preconditions (row sums at most 2^32) at their boundary.
* Algorithm 2 in the ring: stable for every batch cap, coarsest with one
  batch.
"""
import random

import numpy as np
import pytest

import oracle
from oracle import bruteforce as bf

P = (1 << 61) - 1
M64 = (1 << 64) - 1
R = oracle.RING64


def _z(v):
    return [int(x) for x in v]


# ---------------------------------------------------------------------------
# The ring values
# ---------------------------------------------------------------------------

def test_ring_values_unreduced_and_distinct():
    ws = [oracle.weight(7, 3, b, R) for b in range(20000)]
    # residues mod p are the F_p values
    assert all(w % P == oracle.weight(7, 3, b) for b, w in enumerate(ws[:2000]))
    assert len(set(ws)) == len(ws)
    # spread over [0, 2^64): about 7/8 of them are >= 2^61, mean near 2^63
    big = sum(w >= (1 << 61) for w in ws) / len(ws)
    assert abs(big - 7 / 8) < 0.02
    mean = sum(ws) / len(ws) / 2.0**64
    assert abs(mean - 0.5) < 3 * (1 / 12) ** 0.5 / len(ws) ** 0.5


def test_many_colours_one_draw():
    # the repeat-until-distinct condition holds on the first draw even for
    # a round with 300000 colours (every node its own colour)
    n = 300000
    rp = np.arange(n + 1, dtype=np.uint64)
    col = ((np.arange(n, dtype=np.uint64) * 7919) % n).astype(np.uint32)
    c = np.arange(n, dtype=np.uint32)
    z = oracle.image(rp, col, None, c, n, 3, 9, R)
    assert len(set(_z(z))) == n


# ---------------------------------------------------------------------------
# Closed forms of the image
# ---------------------------------------------------------------------------

def test_power_of_two_weights_shift_the_value():
    # rows: [2^31 * w0], [2^31 * w0 + 2^31 * w0] = [2^32 * w0], [1 * w1]
    rp = np.array([0, 1, 3, 4, 4], np.uint64)
    col = np.array([3, 3, 3, 1], np.uint32)
    wt = np.array([1 << 31, 1 << 31, 1 << 31, 1], np.uint32)
    c = np.array([0, 1, 0, 0], np.uint32)
    z = _z(oracle.image(rp, col, wt, c, 2, 4, 1, R))
    w0 = oracle.weight(4, 1, 0, R)
    w1 = oracle.weight(4, 1, 1, R)
    assert z[0] == (w0 << 31) & M64
    assert z[1] == (w0 & 0xFFFFFFFF) << 32  # the top 32 bits of w0 drop out
    assert z[2] == w1
    assert z[3] == 0


def test_long_row_of_largest_weights_wraps():
    rp = np.array([0, 300, 300, 300, 300], np.uint64)
    col = np.array([1, 2, 3] * 100, np.uint32)
    wt = np.full(300, 0xFFFFFFFF, np.uint32)
    c = np.array([0, 1, 2, 3], np.uint32)
    z = _z(oracle.image(rp, col, wt, c, 4, 1, 0, R))
    w = [oracle.weight(1, 0, b, R) for b in range(4)]
    exact = 100 * 0xFFFFFFFF * (w[1] + w[2] + w[3])
    assert exact >= 1 << 90
    assert z[0] == exact % (1 << 64)
    assert z[1:] == [0, 0, 0]


@pytest.mark.parametrize("trial", range(10))
def test_image_linear_over_the_ring(trial):
    # (A + B) w = A w + B w and (2A) w = 2 (A w), both mod 2^64
    rng = random.Random(500 + trial)
    n = rng.randint(2, 60)
    ea = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(1, 5 * n))]
    eb = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(1, 5 * n))]
    wa = [rng.randint(1, 0xFFFFFFFF) for _ in ea]
    wb = [rng.randint(1, 0xFFFFFFFF) for _ in eb]
    c = np.array([rng.randrange(5) for _ in range(n)], np.uint32)

    def csr(edges, wts):
        order = sorted(range(len(edges)), key=lambda t: edges[t][0])
        rp = np.zeros(n + 1, np.uint64)
        for u, _ in edges:
            rp[u + 1] += 1
        rp = np.cumsum(rp).astype(np.uint64)
        col = np.array([edges[t][1] for t in order], np.uint32)
        wt = np.array([wts[t] for t in order], np.uint32)
        return rp, col, wt

    za = _z(oracle.image(*csr(ea, wa), c, 5, trial, 2, R))
    zb = _z(oracle.image(*csr(eb, wb), c, 5, trial, 2, R))
    zab = _z(oracle.image(*csr(ea + eb, wa + wb), c, 5, trial, 2, R))
    assert zab == [(x + y) & M64 for x, y in zip(za, zb)]
    half = [max(1, w // 2) for w in wa]
    zh = _z(oracle.image(*csr(ea, half), c, 5, trial, 2, R))
    zd = _z(oracle.image(*csr(ea + ea, half + half), c, 5, trial, 2, R))
    assert zd == [(2 * x) & M64 for x in zh]


# ---------------------------------------------------------------------------
# Partitions
# ---------------------------------------------------------------------------

def _random_graph(rng, n, directed, weighted, multi):
    edges = []
    for _ in range(rng.randint(0, n * (n - 1) // (1 if directed else 2))):
        u, v = rng.randrange(n), rng.randrange(n)
        if u != v:
            edges.append((u, v))
    if not multi:
        seen, e2 = set(), []
        for u, v in edges:
            key = (u, v) if directed else (min(u, v), max(u, v))
            if key not in seen:
                seen.add(key)
                e2.append((u, v))
        edges = e2
    rp, col = bf.to_csr(n, edges, directed=directed)
    wt = None
    if weighted:
        wt = np.array([rng.randint(1, 4) for _ in range(col.size)], np.uint32)
    return rp, col, wt


@pytest.mark.parametrize("trial", range(40))
def test_ring_bruteforce_random_small(trial):
    rng = random.Random(7000 + trial)
    n = rng.randint(1, 7)
    rp, col, wt = _random_graph(rng, n, trial % 2 == 1, trial % 3 == 2, trial % 5 == 3)
    init = None
    if trial % 4 == 0:
        init = np.array([rng.randint(0, 2) for _ in range(n)], np.uint32)
    A = bf.dense_matrix(rp, col, wt)
    truth = bf.coarsest_stable_partition(A, None if init is None else list(init))
    c, k, r, _, st = oracle.stable_coloring(rp, col, wt, init, seed=trial, q=R)
    _, kb, rb, _, _ = oracle.classic_coloring(rp, col, wt, init)
    assert st == 0
    assert bf.partition_of(c) == truth
    assert k == kb == len(truth) and r == rb


@pytest.mark.parametrize("n", range(2, 14))
def test_ring_path_closed_form(n):
    edges = [(i, i + 1) for i in range(n - 1)]
    rp, col = bf.to_csr(n, edges)
    c, k, _, _, st = oracle.stable_coloring(rp, col, seed=n, q=R)
    assert st == 0 and k == (n + 1) // 2
    assert bf.partition_of(c) == bf.partition_of(bf.path_orbits(n))


@pytest.mark.parametrize("deg", [2, 3, 5])
def test_ring_regular_graphs_one_colour(deg):
    # circulant graph on 40 nodes: i ~ i +- 1..d, regular of degree 2d or 2d-1
    n = 40
    edges = set()
    for i in range(n):
        for s in range(1, deg + 1):
            edges.add((min(i, (i + s) % n), max(i, (i + s) % n)))
    rp, col = bf.to_csr(n, sorted(edges))
    c, k, r, _, st = oracle.stable_coloring(rp, col, seed=deg, q=R)
    assert st == 0 and k == 1 and r == 1


@pytest.mark.parametrize("a,b", [(3, 4), (6, 9)])
def test_ring_grid_orbits(a, b):
    edges = []
    for x in range(a):
        for y in range(b):
            v = x * b + y
            if x + 1 < a:
                edges.append((v, v + b))
            if y + 1 < b:
                edges.append((v, v + 1))
    rp, col = bf.to_csr(a * b, edges)
    c, _, _, _, st = oracle.stable_coloring(rp, col, seed=1, q=R)
    assert st == 0 and bf.partition_of(c) == bf.partition_of(bf.grid_orbits(a, b))


@pytest.mark.parametrize("trial", range(8))
def test_ring_equals_classic_larger(trial):
    rng = random.Random(8100 + trial)
    n = rng.randint(200, 3000)
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(n, 4 * n))]
    directed = trial % 2 == 1
    rp, col = bf.to_csr(n, edges, directed=directed)
    wt = None
    if trial % 3 == 0:
        wt = np.array([rng.choice([1, 2, 1 << 20, 0xFFFFFFFF]) for _ in range(col.size)],
                      np.uint32)
    init = np.array([rng.randint(0, 3) for _ in range(n)], np.uint32) if trial % 4 else None
    if wt is not None and not oracle.ring_preconditions(rp, wt):
        wt = (wt & 0xFFFF).astype(np.uint32)
    c, k, r, _, st = oracle.stable_coloring(rp, col, wt, init, seed=trial, q=R)
    cb, kb, rb, _, _ = oracle.classic_coloring(rp, col, wt, init)
    cf, kf, rf, _, _ = oracle.stable_coloring(rp, col, wt, init, seed=trial)
    assert st == 0
    assert bf.partition_of(c) == bf.partition_of(cb) == bf.partition_of(cf)
    assert k == kb == kf and r == rb == rf


# ---------------------------------------------------------------------------
# Theorem 1's preconditions
# ---------------------------------------------------------------------------

def test_row_sum_bound_at_its_boundary():
    rp = np.array([0, 3, 3], np.uint64)
    col = np.array([1, 1, 1], np.uint32)
    ok = np.array([1 << 31, (1 << 31) - 1, 1], np.uint32)  # sum 2^32
    bad = np.array([1 << 31, (1 << 31) - 1, 2], np.uint32)  # sum 2^32 + 1
    assert oracle.ring_preconditions(rp, ok)
    assert not oracle.ring_preconditions(rp, bad)
    assert oracle.stable_coloring(rp, col, ok, q=R)[4] == 0
    assert oracle.stable_coloring(rp, col, bad, q=R)[4] == 3
    # F_p has no such bound
    assert oracle.stable_coloring(rp, col, bad)[4] == 0
    assert oracle.batched_coloring(rp, col, bad, max_batch=2, q=R)[5] == 3


# ---------------------------------------------------------------------------
# Algorithm 2 in the ring
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("trial", range(6))
def test_ring_batched_stable_and_coarsest_with_one_batch(trial):
    rng = random.Random(9100 + trial)
    n = rng.randint(20, 200)
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(n, 4 * n))]
    rp, col = bf.to_csr(n, edges, directed=trial % 2 == 1)
    wt = np.array([rng.randint(1, 5) for _ in range(col.size)], np.uint32) if trial % 3 else None
    coarsest = oracle.first_occurrence(oracle.classic_coloring(rp, col, wt)[0])[0]
    for cap in (7, 40, col.size):
        c, k, _, _, is_coarsest, st = oracle.batched_coloring(rp, col, wt, seed=trial,
                                                              max_batch=cap, q=R)
        assert st == 0
        assert oracle.is_stable(rp, col, wt, c)
        for b in np.unique(c):  # refines the coarsest stable colouring
            assert len(np.unique(coarsest[c == b])) == 1
        if is_coarsest:
            assert np.array_equal(c, coarsest)
    assert is_coarsest  # one batch holds the whole graph
