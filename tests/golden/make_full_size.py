"""Writes the expected results of the full-size workloads from the CPU oracle.

    python tests/golden/make_full_size.py chunglu rmat27
    python tests/golden/make_full_size.py --ring64 rmat27
    python tests/golden/make_full_size.py --exact chunglu rmat27
    python tests/golden/make_full_size.py rmat28

For each workload: the seeded graph from the shared input generators (built on
the GPU, which produces byte-identical CSRs to the CPU build of the same
generators), then Algorithm 1 run by the oracle round by round from the
trivial partition with seed 0.  Stored per workload in
tests/golden/full_<name>.json: n, nnz, a checksum of the CSR, the colour
count after every round, the round count, the final colour count, the SHA-256
of the final colour array (uint32 little-endian) and the colours of 4096
seeded sample nodes.  With --ring64 the oracle computes in the ring Z/2^64
(Algorithm 1 with precision q = 64) and the file is full_<name>_ring64.json.
With --exact the coarsest stable colouring is computed instead by oracle (b'),
the splitter-based refinement (no rounds, no random weights), and
full_<name>_exact.json stores its colour count and the SHA-256 of its
first-occurrence ids (node 0 has colour 0, each new colour the next id).
The R-MAT scale 28 graph (edge factor 32, 1.68e10 entries) is built into
page-locked host memory by the shared generators, and each oracle round runs
as its two steps (image, then relabel) with a progress line after each; its
file stores no CSR checksum (a pass over 67 GB of column indices in numpy
would take minutes), only n, nnz and the oracle's results.
Nothing here calls the HIP library.
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2607_02603_amd import inputs  # noqa: E402

WORKLOADS = {
    "chunglu": "Chung-Lu n=4e6, 64e6 sampled pairs, exponent 2.1, seed 0",
    "rmat27": "R-MAT scale 27, edge factor 16, (0.57,0.19,0.19,0.05), symmetrised+dedup, seed 0",
    "rmat28": "R-MAT scale 28, edge factor 32, (0.57,0.19,0.19,0.05), symmetrised+dedup, seed 0",
}


def say(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def build(name):
    import torch
    dev = torch.device("cuda:0")
    if name == "rmat28":
        # page-locked host arrays, viewed without a copy
        g = inputs.rmat(28, 32, device=dev, host_out=True)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        return g.row_ptr.numpy().view(np.uint64), g.col.numpy().view(np.uint32)
    g = inputs.chung_lu(device=dev) if name == "chunglu" else inputs.rmat(27, 16, device=dev)
    torch.cuda.synchronize()
    rp = g.row_ptr.cpu().numpy().view(np.uint64)
    col = g.col.cpu().numpy().view(np.uint32)
    del g
    torch.cuda.empty_cache()
    return rp, col


def csr_checksum(rp, col):
    """(sum of col[e] * (e + 1), sum of row_ptr) mod 2^64, computed in chunks."""
    acc = np.uint64(0)
    step = 1 << 27
    with np.errstate(over="ignore"):
        for a in range(0, col.size, step):
            c = col[a:a + step].astype(np.uint64)
            idx = np.arange(a + 1, a + 1 + c.size, dtype=np.uint64)
            acc = acc + np.sum(c * idx, dtype=np.uint64)
        rsum = np.sum(rp, dtype=np.uint64)
    return [int(acc), int(rsum)]


def run(name, q=0):
    say(f"{name}: generating")
    rp, col = build(name)
    n = rp.size - 1
    say(f"{name}: n={n} nnz={col.size}")
    c, k = oracle.canonicalize(None, n)
    hist = []
    r = 0
    while True:
        t0 = time.time()
        if name == "rmat28":
            # the round's two steps, each followed by a progress line
            z = oracle.image(rp, col, None, c, k, 0, r, q)
            say(f"{name}: round {r}: image done ({time.time() - t0:.1f} s)")
            c2, k2 = oracle.relabel(c, z)
            del z
        else:
            c2, k2, _ = oracle.refine_round(rp, col, None, c, k, 0, r, q)
        r += 1
        hist.append(k2)
        say(f"{name}: round {r - 1}: {k} -> {k2} colours ({time.time() - t0:.1f} s)")
        c = c2
        if k2 == k:
            break
        k = k2
    rng = np.random.default_rng(12345)
    sample = np.sort(rng.choice(n, size=min(n, 4096), replace=False)).astype(np.int64)
    out = {
        "workload": WORKLOADS[name], "seed": 0, "n": int(n), "nnz": int(col.size),
        "csr_checksum": None if name == "rmat28" else csr_checksum(rp, col),
        "k_per_round": hist, "rounds": r,
        "colours": int(k), "sha256": hashlib.sha256(c.astype("<u4").tobytes()).hexdigest(),
        "sample_nodes": sample.tolist(), "sample_colours": c[sample].astype(int).tolist(),
        "written_by": "tests/golden/make_full_size.py (oracle/ only)",
    }
    if q:
        out["arithmetic"] = "Z/2^64"
    path = os.path.join(HERE, f"full_{name}{'_ring64' if q else ''}.json")
    with open(path, "w") as f:
        json.dump(out, f)
    say(f"{name}: wrote {path}: colours={k} rounds={r}")


def run_exact(name):
    say(f"{name}: generating")
    rp, col = build(name)
    n = rp.size - 1
    say(f"{name}: n={n} nnz={col.size}; oracle (b') running")
    os.environ["ORC_PROGRESS"] = "1"
    t0 = time.time()
    c, k, visits = oracle.splitter_coloring(rp, col)
    dt = time.time() - t0
    say(f"{name}: colours={k} visits={visits} ({dt:.1f} s)")
    out = {
        "workload": WORKLOADS[name], "n": int(n), "nnz": int(col.size),
        "csr_checksum": csr_checksum(rp, col), "colours": int(k),
        "sha256_first_occurrence": hashlib.sha256(c.astype("<u4").tobytes()).hexdigest(),
        "splitter_visits": int(visits), "seconds": round(dt, 1),
        "written_by": "tests/golden/make_full_size.py --exact (oracle/ only: splitter_coloring)",
    }
    path = os.path.join(HERE, f"full_{name}_exact.json")
    with open(path, "w") as f:
        json.dump(out, f)
    say(f"{name}: wrote {path}")


if __name__ == "__main__":
    args = sys.argv[1:]
    q = oracle.RING64 if "--ring64" in args else oracle.FP
    names = [a for a in args if not a.startswith("--")]
    for nm in names or list(WORKLOADS):
        if "--exact" in args:
            run_exact(nm)
        else:
            run(nm, q)
