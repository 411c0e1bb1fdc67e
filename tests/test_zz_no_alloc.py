"""The allocation-free entry point wl_stable_coloring_noalloc, called through
the C ABI, against wl_stable_coloring with a caller's workspace: identical
colours, colour count and rounds, on consecutive calls whose inputs shrink
(the fixed per-GPU scratch keeps the previous call's contents)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02603_amd as wl
from paper_2607_02603_amd import inputs

pytestmark = pytest.mark.gpu


def _noalloc(dg, init=None, seed=0, max_rounds=0):
    L = wl.lib()
    out = torch.full((dg.n,), -1, dtype=torch.int32, device=dg.device)
    k, r = ctypes.c_uint32(0), ctypes.c_uint32(0)
    s = dg.csr()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    code = L.wl_stable_coloring_noalloc(
        ctypes.byref(s), None if init is None else ctypes.c_void_p(init.data_ptr()), seed,
        max_rounds, ctypes.c_void_p(out.data_ptr()), ctypes.byref(k), ctypes.byref(r), stream)
    torch.cuda.synchronize()
    return code, out, int(k.value), int(r.value)


def _reference(dg, init=None, seed=0):
    c, k, r = wl.wl_stable_coloring(dg, init, seed)
    torch.cuda.synchronize()
    return c, k, r


def _same(dg, init=None, seed=0, label=""):
    print(f"noalloc {label}: n={dg.n} nnz={dg.nnz}", flush=True)
    code, c, k, r = _noalloc(dg, init, seed)
    assert code == wl.WL_OK, wl.lib().wl_last_error()
    rc, rk, rr = _reference(dg, init, seed)
    assert (k, r) == (rk, rr)
    assert torch.equal(c, rc)
    return c, k, r


def test_consecutive_calls_shrinking_inputs():
    big = inputs.rmat(16, 8, seed=1)
    small = inputs.rmat(10, 4, seed=2)
    dbig = wl.Graph.from_numpy(big.n, big.row_ptr, big.col, device="cuda:0")
    dsmall = wl.Graph.from_numpy(small.n, small.row_ptr, small.col, device="cuda:0")
    _same(dbig, label="R-MAT 16")
    c, k, r = _same(dsmall, label="R-MAT 10 after R-MAT 16")
    # the smaller call also equals the oracle bit for bit
    ref, kr, rr, _, st = oracle.stable_coloring(small.row_ptr, small.col)
    assert st == 0 and (k, r) == (kr, rr)
    assert np.array_equal(c.cpu().numpy().view(np.uint32), ref)


def test_consecutive_calls_labels_seeds_symmetric():
    grid = inputs.grid_graph(40, 50)
    er = inputs.er_graph(3000, 9000, seed=4)
    dgrid = wl.Graph.from_numpy(grid.n, grid.row_ptr, grid.col, device="cuda:0",
                                symmetric=True)
    der = wl.Graph.from_numpy(er.n, er.row_ptr, er.col, device="cuda:0")
    lab = torch.from_numpy((np.arange(grid.n) % 3).astype(np.int32)).cuda()
    c, k, r = _same(dgrid, lab, seed=7, label="grid 40x50 with labels")
    _same(der, seed=3, label="ER 3000 after the grid")
    # a round cap stops the call with WL_EMAXROUNDS, as in wl_stable_coloring
    code, c2, k2, r2 = _noalloc(dgrid, lab, seed=7, max_rounds=2)
    assert code == wl.WL_EMAXROUNDS and r2 == 2


def test_graph_beyond_the_scratch_is_refused():
    g = inputs.rmat(20, 4, seed=3)  # about 130 bytes per node: beyond 64 MiB
    dg = wl.Graph.from_numpy(g.n, g.row_ptr, g.col, device="cuda:0")
    code, *_ = _noalloc(dg)
    assert code == wl.WL_EBUDGET
    assert b"scratch" in wl.lib().wl_last_error()
    # and the next call still works
    small = inputs.rmat(9, 4, seed=5)
    _same(wl.Graph.from_numpy(small.n, small.row_ptr, small.col, device="cuda:0"),
          label="R-MAT 9 after a refusal")
