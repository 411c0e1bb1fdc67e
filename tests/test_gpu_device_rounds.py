"""Rounds launched in device-driven groups (no read-back inside a group)
give exactly the oracle's colours, colour count and round count.

WL_HOST_ROUNDS sets how many rounds are host-driven before the groups start
(0: every round is device-driven) and WL_ASYNC_PASSES how many radix passes a
device-driven round runs before it halts for the host to finish it (0: every
round with a class of more than 2048 nodes halts).  A device-driven round whose
splits need the per-colour shift table (more than 4096 of them) halts too.  WL_GRAPH=1 replays the
device-driven rounds from a captured HIP graph.  All are read at every call,
so the cases below switch them per call.
"""
import os
import random

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02603_amd as wl
from oracle import bruteforce as bf
from paper_2607_02603_amd import inputs

pytestmark = pytest.mark.gpu

SETTINGS = [(0, 0), (0, 1), (0, 2), (3, 0), (3, 2)]


@pytest.fixture
def knobs():
    saved = {k: os.environ.get(k) for k in ("WL_HOST_ROUNDS", "WL_ASYNC_PASSES", "WL_GRAPH")}

    def set_(host_rounds, passes, graph=0):
        os.environ["WL_HOST_ROUNDS"] = str(host_rounds)
        os.environ["WL_ASYNC_PASSES"] = str(passes)
        os.environ["WL_GRAPH"] = str(graph)

    yield set_
    for k, v in saved.items():
        if v is None:
            os.environ.pop(k, None)
        else:
            os.environ[k] = v


def _run(rp, col, wt=None, init=None, seed=0, max_rounds=0):
    n = len(rp) - 1
    g = wl.Graph.from_numpy(n, np.asarray(rp, np.uint64), col, wt, device="cuda")
    init_t = None
    if init is not None:
        init_t = torch.from_numpy(np.asarray(init, np.uint32).view(np.int32)).cuda()
    c, k, r = wl.wl_stable_coloring(g, init_t, seed, max_rounds, allow_max_rounds=True)
    torch.cuda.synchronize()
    return c.cpu().numpy().view(np.uint32), k, r


def _same_as_oracle(rp, col, wt=None, init=None, seed=0, max_rounds=0):
    cg, kg, rg = _run(rp, col, wt, init, seed, max_rounds)
    co, ko, ro, _, st = oracle.stable_coloring(rp, col, wt, init, seed, max_rounds)
    assert (kg, rg) == (ko, ro)
    assert np.array_equal(cg, co)
    return kg, rg, st


def _heavy_graph():
    # one class of 10000 leaves (big for the radix passes), hubs of distinct
    # degrees and pendant paths: big classes keep splitting for rounds
    rng = random.Random(11)
    edges = [(0, i) for i in range(1, 10001)]
    n = 10001
    hubs = []
    for h in range(40):
        hub = n
        n += 1
        hubs.append(hub)
        for _ in range(h * 50 + 3):
            edges.append((hub, n))
            n += 1
    for _ in range(3000):
        prev = rng.choice(hubs)
        for _ in range(rng.randint(1, 12)):
            edges.append((prev, n))
            prev = n
            n += 1
    return bf.to_csr(n, edges)


@pytest.mark.parametrize("host_rounds,passes", SETTINGS)
def test_grid_many_rounds(knobs, host_rounds, passes):
    # 100 x 100 grid: 50 rounds, an interior class of thousands of nodes
    knobs(host_rounds, passes)
    g = inputs.grid_graph(100)
    print(f"grid100 host_rounds={host_rounds} passes={passes}", flush=True)
    k, r, st = _same_as_oracle(g.row_ptr, g.col, seed=1)
    assert (k, r, st) == (1275, 50, 0)


@pytest.mark.parametrize("host_rounds,passes", SETTINGS)
def test_big_classes_and_paths(knobs, host_rounds, passes):
    knobs(host_rounds, passes)
    rp, col = _heavy_graph()
    print(f"heavy host_rounds={host_rounds} passes={passes}", flush=True)
    _same_as_oracle(rp, col, seed=3)


@pytest.mark.parametrize("host_rounds,passes", [(0, 0), (0, 1), (3, 2)])
def test_graph_replay(knobs, host_rounds, passes):
    # the device-driven rounds replayed from the captured two-round graphs,
    # with halts (passes 0, 1) that change the parity of the next group
    knobs(host_rounds, passes, graph=1)
    g = inputs.grid_graph(100)
    print(f"graph replay grid100 host_rounds={host_rounds} passes={passes}", flush=True)
    assert _same_as_oracle(g.row_ptr, g.col, seed=1) == (1275, 50, 0)
    rp, col = _heavy_graph()
    _same_as_oracle(rp, col, seed=3)
    for cap in (7, 20):
        k, r, st = _same_as_oracle(g.row_ptr, g.col, seed=2, max_rounds=cap)
        assert r == cap and st == 1


@pytest.mark.parametrize("host_rounds,passes,graph", [(0, 2, 0), (0, 0, 0), (1, 2, 0), (0, 2, 1)])
def test_many_splits_halt_for_the_shift_table(knobs, host_rounds, passes, graph):
    # 60,000 random labels on an R-MAT graph of 2^17 nodes: the first rounds
    # split far more than 4096 classes at once, so a device-driven round
    # halts before the per-colour shift table and the host finishes it
    knobs(host_rounds, passes, graph)
    g = inputs.rmat(17, 8, seed=9)
    init = np.random.default_rng(4).integers(0, 60000, g.n).astype(np.uint32)
    print(f"shift halt host_rounds={host_rounds} passes={passes} graph={graph}", flush=True)
    k, r, st = _same_as_oracle(g.row_ptr, g.col, init=init, seed=5)
    assert st == 0 and r >= 2


@pytest.mark.parametrize("trial", range(8))
def test_random_graphs_device_driven(knobs, trial):
    knobs(trial % 3, trial % 3)
    rng = random.Random(100 + trial)
    n = rng.randint(1, 400)
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(0, 3 * n))]
    rp, col = bf.to_csr(n, edges, directed=trial % 2 == 1)
    wt = None
    if trial % 3 == 1:
        wt = np.array([rng.choice([1, 2, 5]) for _ in range(col.size)], np.uint32)
    init = None
    if trial % 4 == 2:
        init = np.array([rng.choice([4, 9]) for _ in range(n)], np.uint32)
    print(f"random trial {trial} n={n} m={col.size}", flush=True)
    _same_as_oracle(rp, col, wt, init, seed=trial)


@pytest.mark.parametrize("cap", [1, 9, 13, 50])
def test_round_cap_inside_a_group(knobs, cap):
    # the cap falls inside a device-driven group: the state is that of the
    # capped round and later rounds of the group do nothing
    knobs(4, 1)
    g = inputs.grid_graph(100)
    k, r, st = _same_as_oracle(g.row_ptr, g.col, seed=2, max_rounds=cap)
    assert r == cap and st == (0 if cap == 50 else 1)


def test_stats_count_only_rounds_that_ran(knobs):
    knobs(2, 2)
    g = inputs.grid_graph(60)
    dg = wl.Graph.from_numpy(g.n, g.row_ptr, g.col, None, device="cuda")
    wl.wl_stats_enable(3)
    try:
        _, k, r = wl.wl_stable_coloring(dg)
        st = wl.wl_stats_get()
    finally:
        wl.wl_stats_enable(0)
    assert st["rounds"] == r == 30
    launches = sum(st[kind]["launches"] for kind in ("gather", "pb", "uniform"))
    assert launches == r
    assert st["gather"]["ms"] > 0
