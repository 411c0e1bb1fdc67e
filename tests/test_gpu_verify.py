"""GPU stability certificate (wl_verify_stable) against the oracle's exact
certificate (one round of classic refinement splits nothing), on stable
colourings, perturbed ones, rows of every length class (one wave, LDS,
chunked merges), weighted rows and entries of weight 0."""
import random

import numpy as np
import pytest
import torch

import oracle
import paper_2607_02603_amd as wl
from oracle import bruteforce as bf
from paper_2607_02603_amd import inputs

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _graph(rp, col, wt=None, rp64=False):
    n = len(rp) - 1
    rp = np.asarray(rp, dtype=np.uint64)
    if not rp64:
        rp = rp.astype(np.uint32)
    return wl.Graph.from_numpy(n, rp, col, wt, device="cuda")


def _gpu_verify(g, colors, k=None):
    c = np.asarray(colors, np.uint32)
    if k is None:
        k = int(c.max()) + 1 if c.size else 1
    t = torch.from_numpy(c.view(np.int32)).cuda()
    return wl.wl_verify_stable(g, t, k)


def _agree(rp, col, wt, colors, rp64=False, k=None):
    g = _graph(rp, col, wt, rp64)
    got = _gpu_verify(g, colors, k)
    want = oracle.is_stable(rp, col, wt, colors)
    assert got == want
    return got


@pytest.mark.parametrize("trial", range(16))
def test_random_graphs_stable_and_perturbed(trial):
    rng = random.Random(300 + trial)
    n = rng.randint(2, 400)
    directed = trial % 2 == 1
    weighted = trial % 4 >= 2
    edges = [(rng.randrange(n), rng.randrange(n)) for _ in range(rng.randint(0, 5 * n))]
    rp, col = bf.to_csr(n, edges, directed=directed)
    wt = None
    if weighted:
        wt = np.array([rng.choice([0, 1, 2, 7, 0xFFFFFFFF]) for _ in range(col.size)],
                      np.uint32)
    _say(f"trial {trial} n={n} m={col.size} weighted={weighted}")
    c, k, _, _, st = oracle.stable_coloring(rp, col, wt, None, seed=trial)
    assert st == 0
    assert _agree(rp, col, wt, c, rp64=trial % 3 == 0)
    # perturbations: merge two classes, move one node, random colouring
    if k >= 2:
        c2 = c.copy()
        c2[c2 == k - 1] = 0
        _agree(rp, col, wt, c2, k=k)
        c3 = c.copy()
        c3[rng.randrange(n)] = rng.randrange(k)
        _agree(rp, col, wt, c3, k=k)
    c4 = np.array([rng.randrange(3) for _ in range(n)], np.uint32)
    _agree(rp, col, wt, c4, k=3)
    # discrete colouring is always stable
    assert _agree(rp, col, wt, np.arange(n, dtype=np.uint32))


def _hub_graph(rng, degs, palette, weighted=False, mutate=None):
    """Hubs 0..H-1 (one class) with disjoint leaf sets; every hub sees the
    same multiset of leaf colours, in a different order.  Directed: only the
    hub rows have entries."""
    H = len(degs)
    assert len(set(degs)) == 1 or mutate == "lengths"
    base = [rng.randrange(1, palette + 1) for _ in range(max(degs))]
    rows, colors = [], [0] * H
    nxt = H
    for h, d in enumerate(degs):
        cs = base[:d]
        rng.shuffle(cs)
        row = []
        for cval in cs:
            row.append(nxt)
            colors.append(cval)
            nxt += 1
        rows.append(row)
    n = nxt
    if mutate == "one_colour":
        # hub 1's first leaf gets another colour
        leaf = rows[1][0]
        colors[leaf] = (colors[leaf] % palette) + 1
    rp = np.zeros(n + 1, np.uint64)
    for h in range(H):
        rp[h + 1] = rp[h] + len(rows[h])
    rp[H + 1:] = rp[H]
    col = np.array([j for r in rows for j in r], np.uint32)
    return rp, col, np.array(colors, np.uint32)


@pytest.mark.parametrize("deg", [40, 64, 65, 3000, 4096, 4097, 9000, 16384, 70001])
def test_long_rows_every_sort_path(deg):
    rng = random.Random(deg)
    rp, col, c = _hub_graph(rng, [deg] * 3, 20)
    _say(f"hub rows of {deg}")
    assert _agree(rp, col, None, c, rp64=True)
    rp, col, c = _hub_graph(rng, [deg] * 3, 20, mutate="one_colour")
    assert not _agree(rp, col, None, c)
    rp, col, c = _hub_graph(rng, [deg, deg + 1, deg], 20, mutate="lengths")
    assert not _agree(rp, col, None, c)


def test_many_hubs_of_mixed_lengths():
    # one class per length, 3 hubs each: every merge stage runs with rows
    # of different padded lengths side by side
    rng = random.Random(5)
    parts = []
    for d in (5000, 8192, 8193, 20000, 33000):
        parts.append(_hub_graph(rng, [d] * 3, 50))
    # disjoint union with one colour range per part
    rps, cols, cs = [], [], []
    off_n, off_m, off_c = 0, 0, 0
    for rp, col, c in parts:
        rps.append(rp[:-1] + off_m)
        cols.append(col + off_n)
        cs.append(c + off_c)
        off_n += len(rp) - 1
        off_m += int(rp[-1])
        off_c += int(c.max()) + 1
    rp = np.concatenate(rps + [np.array([off_m], np.uint64)])
    col = np.concatenate(cols)
    c = np.concatenate(cs)
    assert _agree(rp, col, None, c)
    c2 = c.copy()
    c2[-1] = c2[-2] if c2[-1] != c2[-2] else c2[-1] + 1
    _agree(rp, col, None, c2, k=int(c.max()) + 2)


def test_weighted_sums_not_multisets():
    # node 0: (b, 1), (b, 1); node 1: (b, 2); node 2: (b, 2), (b', 0)
    rp = np.array([0, 2, 3, 5, 5, 5, 5], np.uint64)
    col = np.array([3, 4, 5, 3, 4], np.uint32)
    wt = np.array([1, 1, 2, 2, 0], np.uint32)
    # b = colour 1 (nodes 3, 5), b' = colour 2 (node 4)... node 0 reaches 3
    # and 4: make 3 and 4 the same colour so that node 0 sees (b, 2)
    c = np.array([0, 0, 0, 1, 1, 1], np.uint32)
    assert _agree(rp, col, wt, c)
    c2 = np.array([0, 0, 0, 1, 2, 1], np.uint32)
    assert not _agree(rp, col, wt, c2)
    # long weighted rows through the chunked merges
    rng = random.Random(9)
    rp, col, c = _hub_graph(rng, [12000] * 2, 30)
    wt = np.array([rng.choice([1, 2, 3]) for _ in range(col.size)], np.uint32)
    wt[int(rp[1]):] = wt[:int(rp[1])][::-1]  # hub 1 weights = hub 0's, reversed...
    # ... with hub 1's leaves in the reversed colour order as well
    c[2 + int(rp[1]):] = c[2:2 + int(rp[1])][::-1]
    assert _agree(rp, col, wt, c)


def test_configs_er_grid():
    for name, g in (("er", inputs.er_graph()), ("grid", inputs.grid_graph(256))):
        dg = _graph(g.row_ptr, g.col)
        colors, k, r = wl.wl_stable_coloring(dg)
        _say(f"{name}: k={k} rounds={r}")
        assert wl.wl_verify_stable(dg, colors, k)
        c = colors.cpu().numpy().view(np.uint32).copy()
        assert oracle.is_stable(g.row_ptr, g.col, None, c)
        # two rounds before the end (the last round only confirms) the
        # colouring is not stable yet
        assert r >= 3
        prev, kp, _ = wl.wl_stable_coloring(dg, max_rounds=r - 2, allow_max_rounds=True)
        assert kp < k
        assert not wl.wl_verify_stable(dg, prev, kp)


def test_errors_and_empty():
    g = inputs.er_graph(1000, 3000, seed=1)
    dg = _graph(g.row_ptr, g.col)
    c = torch.zeros(g.n, dtype=torch.int32, device="cuda")
    with pytest.raises(wl.WlError) as e:
        wl.wl_verify_stable(dg, c, 0)
    assert e.value.code == wl.WL_EINVAL
    with pytest.raises(wl.WlError) as e:
        wl.wl_verify_stable(dg, c, g.n + 1)
    assert e.value.code == wl.WL_EINVAL
    bad = torch.full((g.n,), 7, dtype=torch.int32, device="cuda")
    with pytest.raises(wl.WlError) as e:
        wl.wl_verify_stable(dg, bad, 5)
    assert e.value.code == wl.WL_EINVAL
    need = wl.wl_verify_workspace_size(dg)
    with pytest.raises(wl.WlError) as e:
        wl.wl_verify_stable(dg, c, 1, ws=wl.workspace(need - 512))
    assert e.value.code == wl.WL_EBUDGET
    e0 = _graph(np.zeros(1, np.uint64), np.zeros(0, np.uint32))
    assert wl.wl_verify_stable(e0, torch.zeros(0, dtype=torch.int32, device="cuda"), 0)
    # edgeless graph: any colouring is stable
    e5 = _graph(np.zeros(6, np.uint64), np.zeros(0, np.uint32))
    assert _gpu_verify(e5, np.array([0, 1, 0, 2, 1], np.uint32))
