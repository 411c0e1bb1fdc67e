"""Pins of oracle (b'), the splitter-based exact refinement.

It computes the coarsest stable colouring (Definitions "Stable Coloring" and
"Coarsest Stable Coloring", Section 3) without rounds, by a work list of
splitter classes.  Pinned against:
* exhaustive search over partitions on random small directed, undirected,
  weighted (zero weights too), multi-edge and looped graphs with random
  initial partitions;
* automorphism orbits of trees, grids and paths, and regular graphs (one
  colour);
* oracle (b), the classic round-by-round refinement, on mid-size random,
  weighted, directed and skewed graphs;
* the O(m log n) bound on splitter visits of "all parts but a largest",
  which listing every part would break (a path of 4096 nodes).
"""
import math
import random

import numpy as np
import pytest

import oracle
from oracle import bruteforce as bf
from paper_2607_02603_amd import inputs

from test_oracle_pins import _random_graph, _path, _cycle


def _same(ca, cb):
    return np.array_equal(oracle.first_occurrence(ca)[0], oracle.first_occurrence(cb)[0])


@pytest.mark.parametrize("trial", range(80))
def test_bruteforce_random_small(trial):
    rng = random.Random(7000 + trial)
    n = rng.randint(1, 7)
    directed = trial % 2 == 1
    weighted = trial % 3 == 2
    multi = trial % 5 == 3
    loops = trial % 7 == 4
    rp, col, wt = _random_graph(rng, n, directed, weighted, multi, loops)
    if trial % 8 == 5:  # zero weights: an entry that adds nothing
        wt = np.array([rng.choice([0, 0, 1, 2]) for _ in range(col.size)], np.uint32)
    init = None
    if trial % 4 == 0:
        init = np.array([rng.randint(0, 2) for _ in range(n)], np.uint32)
    A = bf.dense_matrix(rp, col, wt)
    truth = bf.coarsest_stable_partition(A, None if init is None else list(init))
    c, k, _ = oracle.splitter_coloring(rp, col, wt, init)
    assert bf.partition_of(c) == truth and k == len(truth)
    assert np.array_equal(c, oracle.first_occurrence(c)[0])


def test_bruteforce_n9_sample():
    rng = random.Random(77)
    for directed in (False, True):
        rp, col, wt = _random_graph(rng, 9, directed, False, False, False)
        truth = bf.coarsest_stable_partition(bf.dense_matrix(rp, col, wt))
        assert bf.partition_of(oracle.splitter_coloring(rp, col, wt)[0]) == truth


def test_directed_path_uses_out_neighbourhoods():
    # 0 -> 1 -> 2: out-degrees (1, 1, 0), then 0 and 1 differ by where their
    # entry points; in-degrees (0, 1, 1) would split {0} from {1, 2} first.
    rp, col = bf.to_csr(3, [(0, 1), (1, 2)], directed=True)
    assert oracle.splitter_coloring(rp, col)[1] == 3
    # 0 -> 2, 1 -> 2, 3 -> 0: out-degrees all 1 except node 2; coarsest is
    # {0, 1} | {2} | {3} by out-edges, while in-edges would also split 0 from 1
    rp, col = bf.to_csr(4, [(0, 2), (1, 2), (3, 0)], directed=True)
    c, k, _ = oracle.splitter_coloring(rp, col)
    assert k == 3 and c[0] == c[1]


@pytest.mark.parametrize("name", ["cycle9", "complete6", "edgeless5", "petersen", "c3+c4"])
def test_one_colour_graphs(name):
    if name == "cycle9":
        rp, col = _cycle(9)
    elif name == "complete6":
        rp, col = bf.to_csr(6, [(i, j) for i in range(6) for j in range(i + 1, 6)])
    elif name == "edgeless5":
        rp, col = bf.to_csr(5, [])
    elif name == "petersen":
        outer = [(i, (i + 1) % 5) for i in range(5)]
        inner = [(5 + i, 5 + (i + 2) % 5) for i in range(5)]
        spokes = [(i, 5 + i) for i in range(5)]
        rp, col = bf.to_csr(10, outer + inner + spokes)
    else:
        rp, col = bf.to_csr(7, [(0, 1), (1, 2), (2, 0), (3, 4), (4, 5), (5, 6), (6, 3)])
    c, k, _ = oracle.splitter_coloring(rp, col)
    assert k == 1 and not c.any()


@pytest.mark.parametrize("n", [2, 3, 10, 11, 200])
def test_path_orbits(n):
    rp, col = _path(n)
    c, k, _ = oracle.splitter_coloring(rp, col)
    assert k == (n + 1) // 2
    assert bf.partition_of(c) == bf.partition_of(bf.path_orbits(n))


@pytest.mark.parametrize("a,b", [(4, 4), (7, 12), (16, 16), (5, 30)])
def test_grid_orbits(a, b):
    g = inputs.grid_graph(a, b)
    c, k, _ = oracle.splitter_coloring(g.row_ptr, g.col)
    h, w = (a + 1) // 2, (b + 1) // 2
    assert k == (h * (h + 1) // 2 if a == b else h * w)
    assert bf.partition_of(c) == bf.partition_of(bf.grid_orbits(a, b))


@pytest.mark.parametrize("trial", range(15))
def test_random_trees_orbits(trial):
    rng = random.Random(9100 + trial)
    n = rng.randint(2, 80)
    edges = [(i, rng.randrange(i)) for i in range(1, n)]
    if trial % 3 == 0:
        half = n // 2
        edges = [(i, rng.randrange(i)) for i in range(1, half)]
        edges += [(half + u, half + v) for (u, v) in edges]
        edges.append((0, half))
        n = 2 * half
    rp, col = bf.to_csr(n, edges)
    c, _, _ = oracle.splitter_coloring(rp, col)
    assert bf.partition_of(c) == bf.partition_of(bf.tree_orbits(edges, n))


def test_matches_classic_refinement_mid_size():
    rng = np.random.default_rng(3)
    cases = [inputs.er_graph(3000, 6000, seed=1), inputs.er_graph(20000, 80000, seed=0),
             inputs.rmat(scale=12, edge_factor=8, seed=5), inputs.grid_graph(40, 57)]
    for g in cases:
        rp, col = g.row_ptr, g.col
        n = rp.size - 1
        for wt, init in ((None, None),
                         (rng.integers(0, 4, col.size).astype(np.uint32), None),
                         (None, rng.integers(0, 3, n).astype(np.uint32))):
            cb, kb, _, _, st = oracle.classic_coloring(rp, col, wt, init)
            cs, ks, _ = oracle.splitter_coloring(rp, col, wt, init)
            assert st == 0 and ks == kb and _same(cs, cb)
            assert oracle.is_stable(rp, col, wt, cs)


def test_matches_classic_refinement_directed():
    g = inputs.rmat(scale=11, edge_factor=8, seed=2, directed=True)
    cb, kb, _, _, _ = oracle.classic_coloring(g.row_ptr, g.col)
    cs, ks, _ = oracle.splitter_coloring(g.row_ptr, g.col)
    assert ks == kb and _same(cs, cb)


def test_matches_algorithm1():
    g = inputs.chung_lu(n=20000, samples=100000, seed=4)
    ca, ka, _, _, st = oracle.stable_coloring(g.row_ptr, g.col, None, None, 11)
    cs, ks, _ = oracle.splitter_coloring(g.row_ptr, g.col)
    assert st == 0 and ks == ka and _same(cs, ca)


@pytest.mark.parametrize("n", [1024, 4096])
def test_visits_within_m_log_n(n):
    # a path refines from both ends inwards, one class per step; listing
    # every part of every split would read Theta(n^2) entries, the smaller
    # parts only O(m log n)
    rp, col = _path(n)
    m = int(rp[-1])
    c, k, visits = oracle.splitter_coloring(rp, col)
    assert k == n // 2
    assert visits <= m * (math.floor(math.log2(n)) + 2)


def test_empty_and_single():
    c, k, v = oracle.splitter_coloring(np.zeros(1, np.uint64), np.zeros(0, np.uint32))
    assert c.size == 0 and k == 0 and v == 0
    c, k, v = oracle.splitter_coloring(np.zeros(2, np.uint64), np.zeros(0, np.uint32))
    assert list(c) == [0] and k == 1


def test_planted_list_every_part_breaks_the_bound(tmp_path):
    # the visit bound is what tells "all parts but a largest" from "every
    # part": a CPU copy of the oracle with the rule changed must exceed it
    import ctypes
    import os
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = open(os.path.join(os.path.dirname(oracle.__file__), "wl_oracle.c")).read()
    rule = "if ((was_listed || r != big) && !listed[id])"
    assert src.count(rule) == 1
    planted = tmp_path / "planted.c"
    planted.write_text(src.replace(rule, "if (!listed[id])"))
    so = tmp_path / "planted.so"
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", str(so), str(planted)],
                   check=True, capture_output=True)
    lib = ctypes.CDLL(str(so))
    n = 1024
    rp, col = _path(n)
    rp = np.ascontiguousarray(rp, np.uint64)
    col = np.ascontiguousarray(col, np.uint32)
    out = np.empty(n, np.uint32)
    k, visits = ctypes.c_uint32(0), ctypes.c_uint64(0)
    vp = ctypes.c_void_p
    lib.orc_splitter_coloring(ctypes.c_uint64(n), vp(rp.ctypes.data), vp(col.ctypes.data), None,
                              None, vp(out.ctypes.data), ctypes.byref(k), ctypes.byref(visits))
    bound = int(rp[-1]) * (math.floor(math.log2(n)) + 2)
    assert k.value == n // 2  # still the right partition ...
    assert visits.value > bound  # ... at the cost the bound rules out
    assert oracle.splitter_coloring(rp, col)[2] <= bound
