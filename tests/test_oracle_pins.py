"""Pins of the CPU oracle against things other than itself.

* SplitMix64: published outputs of the reference generator (state 0).
* Coarsest stable partitions by exhaustive search (Definitions "Stable
  Coloring" and "Coarsest Stable Coloring"): random small directed,
  undirected, weighted and multi-edge graphs with random initial partitions.
* Closed forms and symmetry orbits: paths, cycles, complete, edgeless,
  stars, complete bipartite graphs, grids, trees (orbit partition), disjoint
  unions of cycles (1-WL cannot tell them apart).
* Invariants of Algorithm 1: nested refinement, order preservation, fixed
  point, permutation equivariance, seed invariance, per-round agreement with
  classic refinement, rounds <= n - k0 + 1, the certificate.
"""
import random

import numpy as np
import pytest

import oracle
from oracle import bruteforce as bf

P = (1 << 61) - 1


# ---------------------------------------------------------------------------
# SplitMix64 and W
# ---------------------------------------------------------------------------

def test_splitmix64_published_outputs():
    # First outputs of SplitMix64 started from state 0 (Steele, Lea, Flood
    # 2014; Vigna's reference splitmix64.c): next() adds the golden gamma,
    # then applies the output mix.
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [oracle.splitmix_nth(0, i) for i in (1, 2, 3)] == expect


def test_weights_canonical_and_distinct():
    ws = [oracle.weight(7, 3, b) for b in range(20000)]
    assert all(0 <= w < P for w in ws)
    assert len(set(ws)) == len(ws)
    # rounds and seeds give different streams
    assert oracle.weight(7, 3, 5) != oracle.weight(7, 4, 5)
    assert oracle.weight(7, 3, 5) != oracle.weight(8, 3, 5)
    # roughly uniform over [0, p): mean within 3 sigma
    mean = sum(ws) / len(ws) / P
    assert abs(mean - 0.5) < 3 * (1 / 12) ** 0.5 / len(ws) ** 0.5


def test_round0_image_is_degree_times_w0():
    # Uniform start: w is the constant W(seed,0,0), so z_i = deg_i * w mod p.
    rp, col = bf.to_csr(6, [(0, 1), (0, 2), (0, 3), (3, 4), (4, 5), (1, 2)])
    z = oracle.image(rp, col, None, np.zeros(6, np.uint32), 1, 11, 0)
    w0 = oracle.weight(11, 0, 0)
    deg = np.diff(rp.astype(np.int64))
    assert [int(v) for v in z] == [(int(d) * w0) % P for d in deg]


def test_image_weighted_rows_and_empty_rows():
    # A = [[0,3,0],[0,0,0],[2,0,5]] with colours (0,1,0): z0 = 3 w1,
    # z1 = 0 (empty row), z2 = 2 w0 + 5 w0 = 7 w0.
    rp = np.array([0, 1, 1, 3], np.uint64)
    col = np.array([1, 0, 2], np.uint32)
    wt = np.array([3, 2, 5], np.uint32)
    z = oracle.image(rp, col, wt, np.array([0, 1, 0], np.uint32), 2, 5, 2)
    w = [oracle.weight(5, 2, b) for b in range(2)]
    assert [int(v) for v in z] == [3 * w[1] % P, 0, 7 * w[0] % P]


def test_image_large_weights_reduce_mod_p():
    # a * w with a near 2^32 and a long row: checks the exact reduction.
    n = 4
    rp = np.array([0, 300, 300, 300, 300], np.uint64)
    col = np.array([1, 2, 3] * 100, np.uint32)
    wt = np.full(300, 0xFFFFFFFF, np.uint32)
    c = np.array([0, 1, 2, 3], np.uint32)
    z = oracle.image(rp, col, wt, c, 4, 1, 0)
    w = [oracle.weight(1, 0, b) for b in range(4)]
    assert int(z[0]) == (100 * 0xFFFFFFFF * (w[1] + w[2] + w[3])) % P
    assert n == 4


# ---------------------------------------------------------------------------
# Relabel definition: rank of (c, z) among distinct pairs
# ---------------------------------------------------------------------------

def test_relabel_rank_of_pairs():
    c = np.array([1, 0, 1, 0, 2, 1], np.uint32)
    z = np.array([9, 5, 3, 5, 0, 9], np.uint64)
    out, k = oracle.relabel(c, z)
    # distinct pairs in order: (0,5) (1,3) (1,9) (2,0)
    assert k == 4
    assert list(out) == [2, 0, 1, 0, 3, 2]


def test_canonicalize_dense_rank():
    out, k = oracle.canonicalize(np.array([70, 5, 70, 9, 5], np.uint32))
    assert k == 3 and list(out) == [2, 0, 2, 1, 0]


# ---------------------------------------------------------------------------
# Brute force on tiny graphs
# ---------------------------------------------------------------------------

def _random_graph(rng, n, directed, weighted, multi, loops):
    edges = []
    m = rng.randint(0, n * (n - 1) // (1 if directed else 2))
    for _ in range(m):
        u, v = rng.randrange(n), rng.randrange(n)
        if u == v and not loops:
            continue
        edges.append((u, v))
    if not multi:
        seen = set()
        e2 = []
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


@pytest.mark.parametrize("trial", range(60))
def test_bruteforce_random_small(trial):
    rng = random.Random(1000 + trial)
    n = rng.randint(1, 7)
    directed = trial % 2 == 1
    weighted = trial % 3 == 2
    multi = trial % 5 == 3
    loops = trial % 7 == 4
    rp, col, wt = _random_graph(rng, n, directed, weighted, multi, loops)
    init = None
    if trial % 4 == 0:
        init = np.array([rng.randint(0, 2) for _ in range(n)], np.uint32)
    A = bf.dense_matrix(rp, col, wt)
    truth = bf.coarsest_stable_partition(A, None if init is None else list(init))
    ca, ka, ra, _, st = oracle.stable_coloring(rp, col, wt, init, seed=trial)
    cb, kb, rb, _, stb = oracle.classic_coloring(rp, col, wt, init)
    assert st == 0 and stb == 0
    assert bf.partition_of(ca) == truth
    assert bf.partition_of(cb) == truth
    assert ka == kb == len(truth)
    assert ra == rb


@pytest.mark.parametrize("trial", range(20))
def test_bruteforce_zero_weight_entries(trial):
    # an entry of weight 0 adds nothing to a_{i,B} (Definition "Stable
    # Coloring"): both oracles must treat it as absent, as brute force does
    rng = random.Random(5000 + trial)
    n = rng.randint(2, 7)
    rp, col, _ = _random_graph(rng, n, trial % 2 == 1, False, trial % 3 == 0, False)
    wt = np.array([rng.choice([0, 0, 1, 2]) for _ in range(col.size)], np.uint32)
    A = bf.dense_matrix(rp, col, wt)
    truth = bf.coarsest_stable_partition(A)
    ca, ka, ra, _, st = oracle.stable_coloring(rp, col, wt, None, seed=trial)
    cb, kb, rb, _, stb = oracle.classic_coloring(rp, col, wt, None)
    assert st == 0 and stb == 0
    assert bf.partition_of(ca) == truth
    assert bf.partition_of(cb) == truth
    assert ka == kb and ra == rb
    assert oracle.is_stable(rp, col, wt, ca)


def test_bruteforce_n9_sample():
    rng = random.Random(99)
    for _ in range(3):
        rp, col, wt = _random_graph(rng, 9, False, False, False, False)
        A = bf.dense_matrix(rp, col, wt)
        truth = bf.coarsest_stable_partition(A)
        ca = oracle.stable_coloring(rp, col, wt)[0]
        assert bf.partition_of(ca) == truth


def test_directed_uses_out_neighbourhoods():
    # 0 -> 1 -> 2 (a directed path): out-degrees (1, 1, 0); nodes 0 and 1
    # differ only after one step.  Coarsest stable = all singletons.  The
    # transpose would give the same count but a different first split.
    rp, col = bf.to_csr(3, [(0, 1), (1, 2)], directed=True)
    c, k, r, hist, _ = oracle.stable_coloring(rp, col)
    assert k == 3 and list(hist) == [2, 3, 3]
    # out-degree split first: {0,1} vs {2}
    c1, k1, _ = oracle.refine_round(rp, col, None, np.zeros(3, np.uint32), 1, 0, 0)
    assert k1 == 2 and c1[0] == c1[1] != c1[2]


# ---------------------------------------------------------------------------
# Closed forms
# ---------------------------------------------------------------------------

def _path(n):
    return bf.to_csr(n, [(i, i + 1) for i in range(n - 1)])


def _cycle(n):
    return bf.to_csr(n, [(i, (i + 1) % n) for i in range(n)])


@pytest.mark.parametrize("n", range(2, 13))
def test_path_closed_form(n):
    rp, col = _path(n)
    c, k, r, _, _ = oracle.stable_coloring(rp, col)
    h = (n + 1) // 2
    assert k == h and r == h
    assert bf.partition_of(c) == bf.partition_of(bf.path_orbits(n))


@pytest.mark.parametrize("name", ["cycle7", "complete6", "edgeless5", "petersen",
                                  "c3+c4"])
def test_one_colour_graphs(name):
    if name == "cycle7":
        rp, col = _cycle(7)
    elif name == "complete6":
        rp, col = bf.to_csr(6, [(i, j) for i in range(6) for j in range(i + 1, 6)])
    elif name == "edgeless5":
        rp, col = bf.to_csr(5, [])
    elif name == "petersen":
        outer = [(i, (i + 1) % 5) for i in range(5)]
        inner = [(5 + i, 5 + (i + 2) % 5) for i in range(5)]
        spokes = [(i, 5 + i) for i in range(5)]
        rp, col = bf.to_csr(10, outer + inner + spokes)
    else:  # a triangle and a 4-cycle: both 2-regular
        rp, col = bf.to_csr(7, [(0, 1), (1, 2), (2, 0), (3, 4), (4, 5), (5, 6), (6, 3)])
    c, k, r, _, _ = oracle.stable_coloring(rp, col)
    assert k == 1 and r == 1 and set(c.tolist()) == {0}


@pytest.mark.parametrize("s", [2, 3, 9])
def test_star(s):
    rp, col = bf.to_csr(s + 1, [(0, i) for i in range(1, s + 1)])
    c, k, r, _, _ = oracle.stable_coloring(rp, col)
    assert k == 2 and r == 2 and len(set(c[1:].tolist())) == 1


@pytest.mark.parametrize("a,b", [(2, 3), (1, 4), (3, 5)])
def test_complete_bipartite(a, b):
    rp, col = bf.to_csr(a + b, [(i, a + j) for i in range(a) for j in range(b)])
    c, k, r, _, _ = oracle.stable_coloring(rp, col)
    assert k == 2 and r == 2


@pytest.mark.parametrize("a", [2, 3, 4, 5, 8, 11, 16])
def test_square_grid(a):
    from paper_2607_02603_amd import inputs
    g = inputs.grid_graph(a)
    c, k, r, _, _ = oracle.stable_coloring(g.row_ptr, g.col)
    h = (a + 1) // 2
    assert k == h * (h + 1) // 2
    assert r == h
    assert bf.partition_of(c) == bf.partition_of(bf.grid_orbits(a, a))


@pytest.mark.parametrize("a,b", [(2, 5), (3, 4), (6, 9), (7, 12)])
def test_rect_grid(a, b):
    from paper_2607_02603_amd import inputs
    g = inputs.grid_graph(a, b)
    c, k, r, _, _ = oracle.stable_coloring(g.row_ptr, g.col)
    assert k == ((a + 1) // 2) * ((b + 1) // 2)
    assert bf.partition_of(c) == bf.partition_of(bf.grid_orbits(a, b))


@pytest.mark.parametrize("trial", range(25))
def test_random_trees_orbits(trial):
    rng = random.Random(5000 + trial)
    n = rng.randint(2, 60)
    edges = [(i, rng.randrange(i)) for i in range(1, n)]
    if trial % 3 == 0:  # make symmetric trees more likely: mirror a subtree
        half = n // 2
        edges = [(i, rng.randrange(i)) for i in range(1, half)]
        edges += [(half + u, half + v) for (u, v) in edges]
        edges.append((0, half))
        n = 2 * half
    rp, col = bf.to_csr(n, edges)
    c, k, r, _, _ = oracle.stable_coloring(rp, col)
    assert bf.partition_of(c) == bf.partition_of(bf.tree_orbits(edges, n))


# ---------------------------------------------------------------------------
# Invariants of Algorithm 1
# ---------------------------------------------------------------------------

def _rounds_trace(rp, col, wt, init, seed):
    c, k = oracle.canonicalize(init, len(rp) - 1)
    trace = [c.copy()]
    r = 0
    while True:
        c2, k2, _ = oracle.refine_round(rp, col, wt, c, k, seed, r)
        trace.append(c2.copy())
        r += 1
        if k2 == k:
            return trace
        c, k = c2, k2


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_round_invariants(seed):
    from paper_2607_02603_amd import inputs
    g = inputs.rmat(10, 8, seed=1)
    trace = _rounds_trace(g.row_ptr, g.col, None, None, seed)
    for prev, cur in zip(trace, trace[1:]):
        # nested: equal new colour -> equal old colour; order preserving
        order = np.lexsort((cur, prev))
        p, q = prev[order], cur[order]
        assert np.all(np.diff(q.astype(np.int64)) >= 0)
        same = q[1:] == q[:-1]
        assert np.all(p[1:][same] == p[:-1][same])
    assert np.array_equal(trace[-1], trace[-2])  # fixed point
    assert len(trace) - 1 <= g.n  # rounds <= n - k0 + 1


def test_seed_invariance_and_cross_oracle():
    from paper_2607_02603_amd import inputs
    g = inputs.er_graph(3000, 7000, seed=3)
    ref = None
    for seed in (0, 1, 2, 3):
        c, k, r, hist, _ = oracle.stable_coloring(g.row_ptr, g.col, seed=seed)
        part = oracle.first_occurrence(c)[0]
        if ref is None:
            ref = (part, k, r, hist)
        assert np.array_equal(part, ref[0]) and k == ref[1] and r == ref[2]
        assert np.array_equal(hist, ref[3])
    cb, kb, rb, hb, _ = oracle.classic_coloring(g.row_ptr, g.col)
    assert np.array_equal(oracle.first_occurrence(cb)[0], ref[0])
    assert rb == ref[2] and np.array_equal(hb, ref[3])


def test_permutation_equivariance():
    from paper_2607_02603_amd import inputs
    g = inputs.rmat(9, 8, seed=4)
    n = g.n
    rng = np.random.default_rng(0)
    pi = rng.permutation(n)  # node i -> pi[i]
    rp = g.row_ptr.astype(np.int64)
    u = np.repeat(np.arange(n), np.diff(rp))
    v = g.col.astype(np.int64)
    keys = (pi[u].astype(np.uint64) << np.uint64(32)) | pi[v].astype(np.uint64)
    h = inputs.csr_from_keys(keys, n)
    c, k, r, _, _ = oracle.stable_coloring(g.row_ptr, g.col, seed=9)
    c2, k2, r2, _, _ = oracle.stable_coloring(h.row_ptr, h.col, seed=9)
    assert k == k2 and r == r2
    assert np.array_equal(c2[pi], c)  # bit-exact colours per node


def test_initial_partition_respected():
    rp, col = _cycle(8)
    init = np.array([5, 5, 1, 5, 5, 5, 5, 5], np.uint32)
    c, k, r, _, _ = oracle.stable_coloring(rp, col, None, init)
    # refines the initial partition and is the mirror-symmetric colouring
    assert c[2] != c[0]
    assert bf.partition_of(c) == bf.coarsest_stable_partition(
        bf.dense_matrix(rp, col), list(init))


def test_certificate_detects_unstable():
    rp, col = _path(3)
    assert not oracle.is_stable(rp, col, None, np.zeros(3, np.uint32))
    assert oracle.is_stable(rp, col, None, np.array([0, 1, 0], np.uint32))
    # a stable but not coarsest colouring also passes (singletons)
    assert oracle.is_stable(rp, col, None, np.arange(3, dtype=np.uint32))


def test_max_rounds_status():
    rp, col = _path(12)
    c, k, r, _, st = oracle.stable_coloring(rp, col, max_rounds=3)
    assert st == 1 and r == 3


def test_empty_graph_and_single_node():
    c, k, r, _, st = oracle.stable_coloring(np.zeros(1, np.uint64), np.zeros(0, np.uint32))
    assert (k, r, st) == (0, 0, 0)
    c, k, r, _, st = oracle.stable_coloring(np.zeros(2, np.uint64), np.zeros(0, np.uint32))
    assert (k, r) == (1, 1) and list(c) == [0]
