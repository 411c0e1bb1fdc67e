"""The segment sorts of the relabel (Algorithm 1, "coarsest partition refining
H on which z is symmetric": the ranks of (c, z) by lexicographic sorting).

A class of 65 to 2048 members is sorted in LDS by a counting sort on ten bits
of z (a workgroup per segment; segments of at most 512 take one wave each
with nine bits when a round has at least 1024 of them); a bucket whose keys
differ is fixed by an insertion sort when it holds at most WL_SORT_FIX keys
(default 32), and the whole segment otherwise goes to a bitonic network.
WL_SORT_FIX=0 sends every segment with a mixed bucket to the network, so
all paths give the oracle's colours, colour count and round count bit for
bit, in F_p and in Z/2^64.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02603_amd as wl
from paper_2607_02603_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture
def sort_fix():
    saved = os.environ.get("WL_SORT_FIX")

    def set_(v):
        os.environ["WL_SORT_FIX"] = str(v)

    yield set_
    if saved is None:
        os.environ.pop("WL_SORT_FIX", None)
    else:
        os.environ["WL_SORT_FIX"] = saved


def _check(rp, col, q, init=None, seed=3):
    n = len(rp) - 1
    g = wl.Graph.from_numpy(n, np.asarray(rp, np.uint64), col, None, device="cuda")
    init_t = None
    if init is not None:
        init_t = torch.from_numpy(np.asarray(init, np.uint32).view(np.int32)).cuda()
    prev = wl.wl_get_precision()
    wl.wl_set_precision(wl.WL_PRECISION_RING64 if q == 64 else wl.WL_PRECISION_FP)
    try:
        c, k, r = wl.wl_stable_coloring(g, init_t, seed)
        torch.cuda.synchronize()
    finally:
        wl.wl_set_precision(prev)
    co, ko, ro, _, st = oracle.stable_coloring(rp, col, None, init, seed, 0,
                                               q=oracle.RING64 if q == 64 else oracle.FP)
    assert st == 0
    assert (k, r) == (ko, ro)
    assert np.array_equal(c.cpu().numpy().view(np.uint32), co)


@pytest.mark.parametrize("fix", [0, 32, 2048])
@pytest.mark.parametrize("q", [61, 64])
def test_rmat_both_sort_paths(sort_fix, fix, q):
    sort_fix(fix)
    g = inputs.rmat(15, 8, seed=5)
    _check(g.row_ptr, g.col, q)


@pytest.mark.parametrize("fix", [0, 32])
def test_grid_with_labels_both_sort_paths(sort_fix, fix):
    # a 150 x 150 grid whose nodes carry 3 labels: classes of a few hundred
    # members with few distinct images
    sort_fix(fix)
    g = inputs.grid_graph(150)
    init = (np.arange(g.n) * 2654435761 % 3).astype(np.uint32)
    _check(g.row_ptr, g.col, 61, init=init)


@pytest.mark.parametrize("fix", [0, 32])
@pytest.mark.parametrize("q", [61, 64])
def test_many_mid_segments_by_wave(sort_fix, fix, q):
    # 2000 labelled classes of 200 nodes over a random graph: every class
    # splits in the first rounds, so a round has well over 1024 segments of
    # 65 to 512 nodes, which one wave each sorts (the canonical start with
    # the images gathered, the later rounds with them materialised); with
    # WL_SORT_FIX=0 a mixed bucket sends its segment to the wave's network
    sort_fix(fix)
    g = inputs.er_graph(400000, 1000000, seed=7)
    init = (np.arange(g.n) // 200).astype(np.uint32)
    print(f"er400k labels q={q} fix={fix}", flush=True)
    _check(g.row_ptr, g.col, q, init=init)
