"""Seeded input generators: structural properties (CPU)."""
import numpy as np
import pytest

from paper_2607_02603_amd import inputs


def _check_simple_symmetric(g):
    rp = g.row_ptr.astype(np.int64)
    n = g.n
    assert rp[0] == 0 and rp[-1] == g.nnz and np.all(np.diff(rp) >= 0)
    u = np.repeat(np.arange(n), np.diff(rp))
    v = g.col.astype(np.int64)
    assert np.all(v < n)
    assert np.all(u != v)  # no self-loops
    key = u * n + v
    assert np.all(np.diff(key) > 0)  # rows sorted, no duplicates
    rkey = np.sort(v * n + u)
    assert np.array_equal(rkey, key)  # symmetric


def test_er_graph():
    g = inputs.er_graph(2000, 5000, seed=1)
    _check_simple_symmetric(g)
    assert g.nnz == 10000
    g2 = inputs.er_graph(2000, 5000, seed=1)
    assert np.array_equal(g.col, g2.col) and np.array_equal(g.row_ptr, g2.row_ptr)
    g3 = inputs.er_graph(2000, 5000, seed=2)
    assert not np.array_equal(g.col, g3.col)


def test_c1_config_shape():
    g = inputs.er_graph()
    _check_simple_symmetric(g)
    assert g.n == 20000 and g.nnz == 160000 and g.row_ptr.dtype == np.uint32


@pytest.mark.parametrize("a,b", [(1, 1), (1, 5), (4, 4), (5, 9)])
def test_grid(a, b):
    g = inputs.grid_graph(a, b)
    _check_simple_symmetric(g)
    assert g.nnz == 2 * ((a - 1) * b + a * (b - 1))
    deg = np.diff(g.row_ptr.astype(np.int64))
    if a >= 2 and b >= 2:
        assert deg.max() <= 4 and deg.min() == 2


def test_grid_1024_entries():
    g = inputs.grid_graph(1024)
    assert g.n == 1048576 and g.nnz == 4190208


def test_rmat_properties():
    g = inputs.rmat(12, 16, seed=0)
    _check_simple_symmetric(g)
    deg = np.diff(g.row_ptr.astype(np.int64))
    assert g.nnz <= 2 * 16 * 4096
    assert deg.max() > 20 * deg.mean()  # heavy-tailed
    g2 = inputs.rmat(12, 16, seed=0)
    assert np.array_equal(g.col, g2.col)


def test_rmat_quadrant_frequencies():
    # raw bit statistics of the sampler: P(source bit = 1) = c + d = 0.24
    g = inputs.rmat(10, 32, seed=3, abcd=(0.25, 0.25, 0.25, 0.25))
    deg = np.diff(g.row_ptr.astype(np.int64))
    assert deg.max() < 6 * deg.mean()  # uniform parameters: no hubs


def test_chung_lu_properties():
    g = inputs.chung_lu(20000, 100000, seed=0)
    _check_simple_symmetric(g)
    deg = np.diff(g.row_ptr.astype(np.int64))
    # weights decrease with the node id: low ids are the hubs
    assert deg[:20].mean() > 10 * deg[-2000:].mean()


def test_alias_table_probabilities():
    thr, alias = inputs.chung_lu_alias(1000, 2.1)
    n = 1000
    w = np.arange(1, n + 1, dtype=np.float64) ** (-1 / 1.1)
    p = w / w.sum()
    # reconstruct the sampling probability of every column from the table
    q = thr.astype(np.float64) / 2**32 / n
    est = q.copy()
    np.add.at(est, alias, (1.0 / n) - q)
    assert np.allclose(est, p, atol=1e-9)


def test_rmat_directed_is_the_forward_half():
    # the directed graph holds one entry u -> v per sample; its symmetrisation
    # is the undirected R-MAT of the same seed
    gd = inputs.rmat(10, 8, seed=3, directed=True)
    gu = inputs.rmat(10, 8, seed=3)
    rp = np.asarray(gd.row_ptr, np.int64)
    u = np.repeat(np.arange(gd.n), np.diff(rp))
    v = gd.col.astype(np.int64)
    assert np.all(u != v)
    both = np.unique(np.concatenate([u * gd.n + v, v * gd.n + u]))
    rpu = np.asarray(gu.row_ptr, np.int64)
    uu = np.repeat(np.arange(gu.n), np.diff(rpu))
    assert np.array_equal(both, np.unique(uu * gu.n + gu.col.astype(np.int64)))
    # not symmetric, and many nodes without out-edges
    assert gd.nnz < gu.nnz
    assert (np.diff(rp) == 0).sum() > (np.diff(rpu) == 0).sum()
