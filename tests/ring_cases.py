"""Inputs for the ring arithmetic (Z/2^64) tests that need more than a
random graph: a weighted graph whose round-0 image puts the value 2^64 - 1
(the largest key) on chosen members of classes of every sort size.

Construction.  Three helper nodes carry the labels 1, 2, 3 (colours 0, 1, 2
after canonicalisation, values w0, w1, w2 in round 0); a member of a group
class points at them with weights a0, a1, a2.  Its image is
a0 w0 + a1 w1 + a2 w2 (mod 2^64).  To hit a target t we pick a2 and solve
a0 w0 + a1 w1 = t - a2 w2 (mod 2^64) with 1 <= a0, a1 < 2^31: a point of a
shifted two-dimensional lattice in a box, found by Gauss reduction of the
lattice basis and Babai rounding with a few neighbours.  The row sum stays
below 2^32 (Theorem 1's bound).  Only the oracle's weight function is used.
"""
import random
from fractions import Fraction

import numpy as np

import oracle

M = 1 << 64


def _gauss_reduce(b1, b2):
    def dot(u, v):
        return u[0] * v[0] + u[1] * v[1]

    while True:
        if dot(b1, b1) > dot(b2, b2):
            b1, b2 = b2, b1
        mu = Fraction(dot(b1, b2), dot(b1, b1))
        r = round(mu)
        if r == 0:
            return b1, b2
        b2 = (b2[0] - r * b1[0], b2[1] - r * b1[1])


def solve_pair(w0, w1, t, lo=1, hi=(1 << 31) - 1):
    """(a0, a1) with a0 w0 + a1 w1 = t (mod 2^64), lo <= a0, a1 <= hi, or
    None.  Needs w0 odd."""
    assert w0 % 2 == 1
    inv = pow(w0, -1, M)
    # lattice of (x, y) with x w0 + y w1 = 0: basis (-w1/w0, 1), (2^64, 0)
    b1, b2 = _gauss_reduce(((-w1 * inv) % M, 1), (M, 0))
    p = ((t * inv) % M, 0)  # one solution
    c = (lo + hi) // 2
    d = (p[0] - c, p[1] - c)
    det = b1[0] * b2[1] - b1[1] * b2[0]
    u = Fraction(d[0] * b2[1] - d[1] * b2[0], det)
    v = Fraction(b1[0] * d[1] - b1[1] * d[0], det)
    for du in range(-3, 4):
        for dv in range(-3, 4):
            iu, iv = round(u) + du, round(v) + dv
            x = p[0] - iu * b1[0] - iv * b2[0]
            y = p[1] - iu * b1[1] - iv * b2[1]
            if lo <= x <= hi and lo <= y <= hi:
                assert (x * w0 + y * w1 - t) % M == 0
                return x, y
    return None


def max_key_graph(group_sizes=(6, 50, 1000, 5000), targets=(2, 5, 20, 50), seed=None):
    """(row_ptr, col, weight, labels, seed, target_nodes): round 0 of
    Algorithm 1 in Z/2^64 gives z = 2^64 - 1 exactly at target_nodes."""
    if seed is None:
        seed = next(s for s in range(1000) if oracle.weight(s, 0, 0, oracle.RING64) % 2)
    w = [oracle.weight(seed, 0, b, oracle.RING64) for b in range(3)]
    assert w[0] % 2 == 1
    rng = random.Random(seed)
    t = M - 1
    sol = None
    while sol is None:
        a2 = rng.randint(1, 1 << 20)
        sol = solve_pair(w[0], w[1], (t - a2 * w[2]) % M)
    a_max = (sol[0], sol[1], a2)
    helpers = [0, 1, 2]
    rows = [[], [], []]
    labels = [1, 2, 3]
    tnodes = []
    node = 3
    for g, (size, nt) in enumerate(zip(group_sizes, targets)):
        for i in range(size):
            if i < nt:
                ws = a_max
                tnodes.append(node)
            else:
                ws = tuple(rng.randint(1, 1 << 30) for _ in range(3))
            rows.append(list(zip(helpers, ws)))
            labels.append(10 + g)
            node += 1
    # the members are shuffled so the targets do not sit together
    order = list(range(3, node))
    rng.shuffle(order)
    perm = list(range(3)) + order  # new id -> old id
    newid = {old: new for new, old in enumerate(perm)}
    rp = [0]
    col, wt, lab = [], [], []
    for old in perm:
        for h, a in rows[old]:
            col.append(h)
            wt.append(a)
        rp.append(len(col))
        lab.append(labels[old])
    tn = sorted(newid[x] for x in tnodes)
    return (np.array(rp, np.uint64), np.array(col, np.uint32), np.array(wt, np.uint32),
            np.array(lab, np.uint32), seed, tn)
