"""The one-colour round (the degree round of the HIP path) against the oracle.

An unweighted graph that starts from one colour gets its first round from a
degree histogram: the image is z_i = deg_i W (Section 4.1), and the new
colours are the ranks of the distinct values.  The member list of the next
round is written in two parts: class index and row length over each class's
range in position order, the members and their row starts by placement.  A
rank shared by several degrees (values d W that coincide) has members of
different row lengths, which the placement then writes one by one.  Such
ranks need a degenerate W; tests/weight_seeds.py makes the seeds that give
one (2^(64 - j) in Z/2^64: degrees equal mod 2^j share a rank; 0 in F_p: one
rank, no split).  Compared with the oracle in the same arithmetic: colour
ids, colour count and rounds, bit for bit.  The graphs have at least 8,193
nodes, where the degree round applies, and odd sizes for ragged ends.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_02603_amd as wl
from paper_2607_02603_amd import inputs

import weight_seeds as ws

pytestmark = pytest.mark.gpu


@pytest.fixture
def precision():
    prev = wl.wl_get_precision()
    yield wl.wl_set_precision
    wl.wl_set_precision(prev)


def _run(g, seed, q):
    print(f"  n={g.n} nnz={len(g.col)} seed={seed:#x} q={q}", flush=True)
    dg = wl.Graph.from_numpy(g.n, np.asarray(g.row_ptr), g.col, None, device="cuda")
    c, k, r = wl.wl_stable_coloring(dg, None, seed)
    torch.cuda.synchronize()
    got = c.cpu().numpy().view(np.uint32)
    co, ko, ro, _, st = oracle.stable_coloring(g.row_ptr, g.col, None, None, seed, q=q)
    assert st == 0
    assert (k, r) == (ko, ro)
    assert np.array_equal(got, co)
    return k, r


@pytest.mark.parametrize("j", [1, 2, 5])
@pytest.mark.parametrize("graph", ["rmat14", "grid101"])
def test_ring_shared_ranks(precision, j, graph):
    precision(wl.WL_PRECISION_RING64)
    g = inputs.rmat(14, 8, seed=3) if graph == "rmat14" else inputs.grid_graph(101, 103)
    deg = np.diff(np.asarray(g.row_ptr, dtype=np.int64))
    seed = ws.seed_for_weight0(1 << (64 - j))
    shared = len(np.unique(deg)) > len(np.unique(deg % (1 << j)))
    print(f"{graph} j={j} shared ranks: {shared}", flush=True)
    k, r = _run(g, seed, oracle.RING64)
    # the partition is still the coarsest stable one
    cc, kc, _, _, _ = oracle.classic_coloring(g.row_ptr, g.col)
    assert k == kc


def test_fp_zero_weight_one_colour(precision):
    precision(wl.WL_PRECISION_FP)
    g = inputs.rmat(14, 8, seed=3)
    k, r = _run(g, ws.seed_for_weight0(0), oracle.FP)
    assert (k, r) == (1, 1)


@pytest.mark.parametrize("n", [8193, 8195, 9001, 20011])
def test_sizes_around_the_degree_round(precision, n):
    # isolated nodes (degree 0, not live) and live classes of every size;
    # the member list's length is not a multiple of four
    precision(wl.WL_PRECISION_FP)
    g = inputs.er_graph(n, n, seed=n)
    for seed in (1, 2):
        _run(g, seed, oracle.FP)
