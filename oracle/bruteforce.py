"""Brute force and independent structure for pinning the oracle (tests only).

Nothing here runs the refinement method.  These are other, independent ways
to obtain the coarsest stable colouring (Definitions "Stable Coloring" and
"Coarsest Stable Coloring", Section 3) on inputs small or structured enough:

* ``coarsest_stable_partition``: enumerate every partition that refines the
  initial one, keep the stable ones, return the coarsest (n <= 9).
* ``tree_orbits``: automorphism orbits of a tree (canonical rooted-tree
  codes from the centre).  For trees, colour refinement reaches exactly the
  orbit partition, a classical fact about trees.
* ``grid_orbits`` / ``path_orbits``: orbits of the symmetry group of an
  a x b grid (the dihedral group of the rectangle) and of a path.
"""
from itertools import product

import numpy as np


def dense_matrix(row_ptr, col, weight=None):
    n = len(row_ptr) - 1
    A = [[0] * n for _ in range(n)]
    for i in range(n):
        for e in range(int(row_ptr[i]), int(row_ptr[i + 1])):
            A[i][int(col[e])] += 1 if weight is None else int(weight[e])
    return A


def is_stable_partition(A, blocks):
    """Definition "Stable Coloring": equal out-weight into every block."""
    for B in blocks:
        for Bp in blocks:
            sums = {sum(A[i][l] for l in Bp) for i in B}
            if len(sums) > 1:
                return False
    return True


def _set_partitions(items):
    if not items:
        yield []
        return
    first, rest = items[0], items[1:]
    for part in _set_partitions(rest):
        yield [[first]] + part
        for t in range(len(part)):
            yield part[:t] + [[first] + part[t]] + part[t + 1:]


def coarsest_stable_partition(A, init=None):
    """The coarsest stable partition refining the initial one (as a list of
    sorted blocks), by exhaustive search.  It is unique; the search also
    asserts that it is coarser than every other stable partition found."""
    n = len(A)
    if n == 0:
        return []
    labels = [0] * n if init is None else list(init)
    groups = {}
    for i, l in enumerate(labels):
        groups.setdefault(l, []).append(i)
    per_group = [list(_set_partitions(g)) for g in groups.values()]
    stable = []
    for combo in product(*per_group):
        blocks = [b for part in combo for b in part]
        if is_stable_partition(A, blocks):
            stable.append(blocks)
    best = min(stable, key=len)
    best_of = {}
    for bi, b in enumerate(best):
        for i in b:
            best_of[i] = bi
    for other in stable:  # every stable partition refines the coarsest one
        for b in other:
            assert len({best_of[i] for i in b}) == 1
    return sorted(sorted(b) for b in best)


def partition_of(colors):
    """Partition (sorted list of sorted blocks) induced by a colour vector."""
    blocks = {}
    for i, c in enumerate(colors):
        blocks.setdefault(int(c), []).append(i)
    return sorted(sorted(b) for b in blocks.values())


def _tree_centres(adj):
    n = len(adj)
    if n <= 2:
        return list(range(n))
    deg = [len(a) for a in adj]
    leaves = [i for i in range(n) if deg[i] <= 1]
    removed = len(leaves)
    while removed < n:
        nxt = []
        for v in leaves:
            for u in adj[v]:
                deg[u] -= 1
                if deg[u] == 1:
                    nxt.append(u)
        removed += len(nxt)
        if removed >= n:
            return nxt
        leaves = nxt
    return leaves


def _rooted_codes(adj, root):
    """Canonical code of the subtree hanging from every node (rooted at
    'root'), AHU style: a node's code is the sorted tuple of its children's
    codes."""
    n = len(adj)
    parent = [-1] * n
    order = [root]
    parent[root] = root
    for v in order:
        for u in adj[v]:
            if parent[u] == -1:
                parent[u] = v
                order.append(u)
    code = [None] * n
    for v in reversed(order):
        kids = sorted(code[u] for u in adj[v] if parent[u] == v and u != v)
        code[v] = tuple(kids)
    return code, parent, order


def tree_orbits(edges, n):
    """Automorphism orbits of a tree on n nodes given by its edge list."""
    adj = [[] for _ in range(n)]
    for u, v in edges:
        adj[u].append(v)
        adj[v].append(u)
    cs = _tree_centres(adj)
    if len(cs) == 1:
        code, parent, order = _rooted_codes(adj, cs[0])
        root_codes = {cs[0]: code[cs[0]]}
    else:
        # bicentral: root at the centre edge; both halves are compared
        a, b = cs
        adj2 = [list(x) for x in adj]
        adj2[a].remove(b)
        adj2[b].remove(a)
        ca, _, _ = _rooted_codes(adj2, a)
        cb, _, _ = _rooted_codes(adj2, b)
        code = [ca[i] if ca[i] is not None else cb[i] for i in range(n)]
        # nodes on the two sides are equivalent iff the halves are isomorphic
        swap = ca[a] == cb[b]
        side = [None] * n
        stack = [(a, 0), (b, 1)]
        seen = {a, b}
        while stack:
            v, s = stack.pop()
            side[v] = s
            for u in adj2[v]:
                if u not in seen:
                    seen.add(u)
                    stack.append((u, s))
    # orbit key: the code of the node together with the codes of the path to
    # the root (the chain of ancestors' codes identifies the position).
    if len(cs) == 1:
        key = []
        for v in range(n):
            chain = []
            w = v
            while True:
                chain.append(code[w])
                if w == parent[w]:
                    break
                w = parent[w]
            key.append(tuple(chain))
    else:
        a, b = cs
        _, pa, _ = _rooted_codes(adj2, a)
        _, pb, _ = _rooted_codes(adj2, b)
        key = []
        for v in range(n):
            par = pa if side[v] == 0 else pb
            chain = []
            w = v
            while True:
                chain.append(code[w])
                if w == par[w]:
                    break
                w = par[w]
            tag = 0 if swap else side[v]
            key.append((tag, tuple(chain)))
    ids = {}
    return [ids.setdefault(k, len(ids)) for k in key]


def grid_orbits(a, b):
    """Orbit id of every cell of the a x b grid (id = r * b + s) under the
    grid's symmetry group (reflections, and the diagonal ones when a == b)."""
    out = []
    ids = {}
    for r in range(a):
        for s in range(b):
            rr = min(r, a - 1 - r)
            ss = min(s, b - 1 - s)
            key = tuple(sorted((rr, ss))) if a == b else (rr, ss)
            out.append(ids.setdefault(key, len(ids)))
    return out


def path_orbits(n):
    ids = {}
    return [ids.setdefault(min(i, n - 1 - i), len(ids)) for i in range(n)]


def to_csr(n, edges, directed=False):
    """CSR (row_ptr uint64, col uint32) of an edge list; undirected edges are
    stored in both directions; duplicates are kept (multi-edges)."""
    rows = [[] for _ in range(n)]
    for u, v in edges:
        rows[u].append(v)
        if not directed and u != v:
            rows[v].append(u)
    rp = np.zeros(n + 1, dtype=np.uint64)
    for i in range(n):
        rp[i + 1] = rp[i] + len(rows[i])
    col = np.array([v for r in rows for v in sorted(r)], dtype=np.uint32)
    return rp, col
