"""A chained scan of the incremental rounds gives up after a bounded wait.

The classes that split in a round are listed in colour order by a chained
scan (decoupled look-back) over chunks of 256 live classes: a chunk waits for
an earlier one at most WL_CHAIN_SPINS polls (read at every call; the default
is far beyond any real wait).  With the bound at 0, a call whose chunks never
had to wait completes with the usual colouring, and a call where one had to
wait stops the device and fails with WL_EHIP: it never returns a different
result.  A following call with the default bound gives the exact colouring
again.  Only the host-set bound is forced: every kernel exits normally.

The a x a grid's coarsest colouring has ceil(a/2)(ceil(a/2)+1)/2 colours,
reached in ceil(a/2) rounds (the dihedral orbits; tests/test_oracle_pins.py
pins the oracle to them); the 100 x 100 case is also compared with the
oracle colour by colour.
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
def spins():
    saved = os.environ.get("WL_CHAIN_SPINS")

    def set_(v):
        if v is None:
            os.environ.pop("WL_CHAIN_SPINS", None)
        else:
            os.environ["WL_CHAIN_SPINS"] = str(v)

    yield set_
    if saved is None:
        os.environ.pop("WL_CHAIN_SPINS", None)
    else:
        os.environ["WL_CHAIN_SPINS"] = saved


def _call(g, seed):
    """(colours, k, rounds), or None when the call gave up with WL_EHIP."""
    dg = wl.Graph.from_numpy(g.n, np.asarray(g.row_ptr, np.uint64), g.col, None, device="cuda")
    try:
        c, k, r = wl.wl_stable_coloring(dg, None, seed)
    except wl.WlError as e:
        assert e.code == wl.WL_EHIP and "chained scan" in str(e), str(e)
        print("  gave up:", e, flush=True)
        return None
    torch.cuda.synchronize()
    print(f"  completed: k={k} rounds={r}", flush=True)
    return c.cpu().numpy().view(np.uint32), k, r


def _grid_closed_form(a):
    h = (a + 1) // 2
    return h * (h + 1) // 2, h


def test_zero_bound_against_oracle(spins):
    g = inputs.grid_graph(100)
    co, ko, ro, _, _ = oracle.stable_coloring(g.row_ptr, g.col, None, None, 2, 0)
    assert (ko, ro) == _grid_closed_form(100)
    spins(0)
    print("grid100 WL_CHAIN_SPINS=0", flush=True)
    got = _call(g, 2)
    if got is not None:
        assert (got[1], got[2]) == (ko, ro)
        assert np.array_equal(got[0], co)
    spins(None)
    print("grid100 default bound", flush=True)
    c, k, r = _call(g, 2)
    assert (k, r) == (ko, ro)
    assert np.array_equal(c, co)


def test_zero_bound_many_chunks(spins):
    # 256 x 256: up to 8256 live classes, 33 chunks a round, 128 rounds
    g = inputs.grid_graph(256)
    kk, rr = _grid_closed_form(256)
    spins(0)
    print("grid256 WL_CHAIN_SPINS=0", flush=True)
    first = _call(g, 5)
    spins(None)
    print("grid256 default bound", flush=True)
    c, k, r = _call(g, 5)
    assert (k, r) == (kk, rr)
    if first is not None:
        assert (first[1], first[2]) == (k, r)
        assert np.array_equal(first[0], c)
