"""Algorithm 1 on the oracle when the weight of round 0 is degenerate.

Seeds from tests/weight_seeds.py give the single colour of round 0 a chosen
weight W; they are checked here against the oracle's weight function, which
test_oracle_pins.py ties to SplitMix64's published outputs.  With one colour
the image of an unweighted graph is z_i = deg_i W (Section 4.1), so:

* in Z/2^64 with W = 2^(64 - j), z_i = (deg_i mod 2^j) 2^(64 - j): after one
  round the colours are the dense ranks of deg_i mod 2^j, and degrees that
  agree mod 2^j share a colour;
* in F_p with W = 0 every image is 0, no class splits, and Algorithm 1 stops
  after that round with the single colour (the failure that its error bound
  allows, here forced).

After the degenerate round the weights are ordinary again: the ring runs go
on to the coarsest stable colouring, classic refinement's partition.
"""
import random

import numpy as np
import pytest

import oracle
from paper_2607_02603_amd import inputs

import weight_seeds as ws

R = oracle.RING64
FP = oracle.FP


def test_mix_matches_the_oracle():
    rng = random.Random(11)
    for _ in range(2000):
        z = rng.getrandbits(64)
        assert ws.mix(z) == oracle.mix64(z)
        assert ws.unmix(ws.mix(z)) == z


@pytest.mark.parametrize("w", [1 << 62, 1 << 63, 1 << 59, 3 << 40, 0, 1, (1 << 64) - 1])
def test_seed_gives_the_chosen_weight(w):
    seed = ws.seed_for_weight0(w)
    assert oracle.weight(seed, 0, 0, R) == w
    # in F_p the weight is the residue of the same word
    assert oracle.weight(seed, 0, 0, FP) == w % ((1 << 61) - 1)
    # only colour 0 of round 0 is chosen: the next values are ordinary
    assert oracle.weight(seed, 0, 1, R) not in (0, w)
    assert oracle.weight(seed, 1, 0, R) not in (0, w)


def _degrees(g):
    return np.diff(np.asarray(g.row_ptr, dtype=np.int64))


@pytest.mark.parametrize("j", [1, 2, 5])
def test_ring_round0_ranks_degrees_mod_power_of_two(j):
    g = inputs.rmat(10, 8, seed=3)
    deg = _degrees(g)
    assert (deg == 0).any() and len(np.unique(deg)) > 2 ** j
    seed = ws.seed_for_weight0(1 << (64 - j))
    c, k, r, hist, st = oracle.stable_coloring(g.row_ptr, g.col, None, None, seed, 1, q=R)
    vals, expect = np.unique(deg % (1 << j), return_inverse=True)
    assert (k, r) == (len(vals), 1)
    assert np.array_equal(c, expect.astype(np.uint32))


@pytest.mark.parametrize("j", [1, 2])
def test_ring_degenerate_round_then_coarsest(j):
    g = inputs.rmat(10, 8, seed=4)
    seed = ws.seed_for_weight0(1 << (64 - j))
    c, k, r, hist, st = oracle.stable_coloring(g.row_ptr, g.col, None, None, seed, q=R)
    cc, kc, rc, _, stc = oracle.classic_coloring(g.row_ptr, g.col)
    assert st == 0 and stc == 0
    assert k == kc
    assert np.array_equal(oracle.first_occurrence(c)[0], oracle.first_occurrence(cc)[0])
    # round 0 merged degrees that differ: fewer colours than the degree partition
    assert hist[0] < len(np.unique(_degrees(g)))


def test_fp_zero_weight_stops_with_one_colour():
    g = inputs.rmat(10, 8, seed=3)
    seed = ws.seed_for_weight0(0)
    c, k, r, hist, st = oracle.stable_coloring(g.row_ptr, g.col, None, None, seed, q=FP)
    assert st == 0 and k == 1 and r == 1
    assert not c.any()
