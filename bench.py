"""Benchmark: randomized 1-WL stable colouring on one MI355X.

A step is one whole call of wl_stable_coloring (canonical start, every
SpMV + relabel round, the confirming round) on a graph already resident in
HBM.  Default workload: undirected R-MAT scale 27, edge factor 16,
(a, b, c, d) = (0.57, 0.19, 0.19, 0.05), symmetrised and deduplicated,
uint64 row pointers, generated on the GPU from seed 0.

Prints one JSON line: GTEPS per refinement round (directed CSR entries x
rounds / time-to-stable), time-to-stable in ms_per_step, the roofline of the
dominant image launch (the step "z = A w" of a round; on R-MAT scale 27 the
propagation-blocking image of the full round) and the CPU oracle timed on a
bounded sample.  The roofline's HBM traffic comes from the rocprofv3 counter
summary under profiles/ when it was taken on the current kernel source.
config also carries the rate of the CSR entries the image launches actually
read (active_edge_gteps: rows of classes that cannot split are skipped), the
measured HBM traffic of the whole call over its kernel time (call_traffic,
from the counter summary of all library kernels, when it matches the current
sources), and, in the untimed run, whether the colour array equals the
oracle's stored result for the workload (check).
"""
import argparse
import json
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0

WORKLOADS = {
    "er": dict(desc="Erdos-Renyi G(n=20000, m=80000), seed 0"),
    "grid": dict(desc="2D grid 1024x1024, 4-neighbour"),
    "chunglu": dict(desc="Chung-Lu n=4e6, 64e6 sampled pairs, exponent 2.1, seed 0"),
    "rmat27": dict(desc="R-MAT scale 27, edge factor 16, (0.57,0.19,0.19,0.05), "
                        "symmetrised+dedup, seed 0"),
    "rmat28b": dict(desc="R-MAT scale 28, edge factor 32, (0.57,0.19,0.19,0.05), "
                         "symmetrised+dedup, seed 0, CSR in pinned host memory, "
                         "under a 32 GiB device workspace"),
    "rmat29s": dict(desc="R-MAT scale 29, edge factor 32, (0.57,0.19,0.19,0.05), "
                         "symmetrised+dedup, seed 0, CSR in pageable host memory, "
                         "streamed workspace plus 8 GiB"),
}

# Arithmetic of the image step (--arith): the prime field of the default
# path, or the ring of Section 4.1 (Algorithm 1 with precision q = 64).
ARITH = {"fp": (0, "F_p, p = 2^61 - 1"), "ring64": (64, "Z/2^64")}

# How the out-of-core workload is refined (--batched-mode):
#   plain        Algorithm 2 as printed (outer loop to its fixed point)
#   exact        Algorithm 2, then the exact finish (Algorithm 1 streamed)
#   exact-early  Section 5.4's early stop, then the exact finish
#   streamed     Algorithm 1 with the image streamed from host memory
BATCHED_MODES = {
    "plain": "batched (Algorithm 2, outer loop to its fixed point)",
    "exact": "batched (Algorithm 2 to its fixed point) + exact streamed finish",
    "exact-early": "batched (Algorithm 2, early stop of Section 5.4) + exact streamed finish",
    "streamed": "Algorithm 1 with the image streamed from host memory (no batching)",
}


def bench_batched(args):
    """Out of core: R-MAT scale 28 held in pinned host memory under 32 GiB of
    device workspace (Algorithm 2 or the streamed Algorithm 1), or R-MAT
    scale 29 (over 3e10 entries) in pageable host memory, streamed, with the
    workspace that mode asks for; optionally checked against the in-core
    colouring of the same graph copied to HBM."""
    import torch
    import paper_2607_02603_amd as wl
    from paper_2607_02603_amd import inputs
    dev = torch.device("cuda:0")
    big = args.workload == "rmat29s"
    if big and args.batched_mode != "streamed":
        raise SystemExit("rmat29s runs the streamed mode only")
    if args.batched_mode in ("exact", "exact-early"):
        # the library accepts WL_BATCHED_EXACT only up to 2^31 entries, far
        # below these graphs: say so before building them
        raise SystemExit(f"--batched-mode {args.batched_mode} is switched off for "
                         f"{args.workload}: the library's exact finish is limited to "
                         f"2^31 entries (use --batched-mode streamed)")
    t0 = time.perf_counter()
    if big:
        g = inputs.rmat(29, 32, device=dev, host_out=True, pinned=False)
    else:
        g = inputs.rmat(28, 32, device=dev, host_out=True)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log(f"graph {args.workload} (host): n={g.n} nnz={g.nnz} built in "
        f"{time.perf_counter() - t0:.1f}s")
    hg = wl.Graph(g.n, g.row_ptr, g.col)
    # R-MAT 29: the streamed mode's workspace and 8 GiB more, in which the
    # rounds after the full one keep their chunks on the device
    ws = wl.workspace(wl.wl_streamed_workspace_size(hg) + (8 << 30) if big else 32 << 30, dev)
    mode = args.batched_mode
    opts = {"plain": 0, "exact": wl.WL_BATCHED_EXACT,
            "exact-early": wl.WL_BATCHED_EXACT | wl.WL_BATCHED_EARLY_STOP}.get(mode)
    res = None
    times = []
    for i in range(args.warmup + args.steps):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        if mode == "streamed":
            # raw rank ids, the same as the in-core call's
            c, kk, rr = wl.wl_stable_coloring_streamed(hg, None, 0, ws=ws)
            res = (c, kk, rr, 0, True)
        else:
            res = wl.wl_stable_coloring_batched(hg, None, 0, 0, ws=ws, options=opts)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t1
        if i >= args.warmup:
            times.append(dt)
        log(f"{'warmup' if i < args.warmup else 'step'} {i}: {dt * 1e3:.1f} ms "
            f"colours={res[1]} rounds={res[2]} outer={res[3]} coarsest={res[4]}")
    colors, k, rounds, outer, coarsest = res
    step_s = sum(times) / len(times)
    check = None
    if args.verify:
        del ws
        torch.cuda.empty_cache()
        dg = wl.Graph(g.n, g.row_ptr.to(dev), g.col.to(dev))
        c_in, k_in, r_in = wl.wl_stable_coloring(dg)
        # first-occurrence relabel of the in-core colours, on the device
        n = g.n
        first = torch.full((k_in,), n, dtype=torch.int64, device=dev)
        idx = torch.arange(n, dtype=torch.int64, device=dev)
        first.scatter_reduce_(0, c_in.long(), idx, reduce="amin")
        order = torch.argsort(first)
        rank = torch.empty_like(order)
        rank[order] = torch.arange(k_in, dtype=torch.int64, device=dev)
        canon = rank[c_in.long()].to(torch.int32)
        if mode == "streamed":
            # the streamed rounds are those of the in-core call: raw ids equal
            same = bool(torch.equal(c_in.cpu(), colors)) and (k, rounds) == (k_in, r_in)
            refines = same
        else:
            bc = colors.to(dev).long()
            # every batched class lies inside one in-core class (the batched
            # colouring refines the coarsest one); equal when the last outer
            # iteration had a single batch or the exact finish ran
            lo = torch.full((k,), k_in, dtype=torch.int64, device=dev)
            hi = torch.full((k,), -1, dtype=torch.int64, device=dev)
            lo.scatter_reduce_(0, bc, canon.long(), reduce="amin")
            hi.scatter_reduce_(0, bc, canon.long(), reduce="amax")
            refines = bool(torch.equal(lo, hi))
            same = bool(torch.equal(canon.cpu(), colors))
        check = {"in_core_colours": k_in, "in_core_rounds": r_in,
                 "batched_refines_in_core": refines, "batched_equals_in_core": same,
                 "excess_colours_frac": (k - k_in) / max(k_in, 1)}
        log(f"in-core: colours={k_in} rounds={r_in}; batched refines in-core: {refines}; "
            f"equal: {same}")
    out = {
        "metric": "time-to-stable-coloring, out-of-core, edges per second",
        "value": g.nnz / step_s / 1e9, "unit": "GTEPS (nnz / time-to-stable)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": step_s * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload]["desc"] + ", " + BATCHED_MODES[mode],
                   "mode": mode, "arithmetic": ARITH[args.arith][1], "n": g.n, "nnz": g.nnz,
                   "colours": k, "rounds_summed_over_batches": rounds,
                   "outer_iterations": outer, "coarsest": coarsest,
                   "time_to_stable_ms": step_s * 1e3, "check": check},
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


STUDY_GRAPHS = {
    "rmat20": "R-MAT scale 20, edge factor 16, undirected (social-like)",
    "rmat20dir": "R-MAT scale 20, edge factor 16, directed (web-like: skewed out- and "
                 "in-degrees, many nodes without out-edges)",
    "chunglu1m": "Chung-Lu n=1e6, 16e6 sampled pairs, exponent 2.1, undirected",
    "rmat22": "R-MAT scale 22, edge factor 16, undirected",
}


def study_reduction(args):
    """Reduction quality of Algorithm 2 (Section 5, Table 1's layout) on
    synthetic graphs: colours as a fraction of n for N_b = 1, 2, 4 batches
    (cap M_b = ceil(m / N_b)), with the outer loop run to its fixed point
    and with the early stop of Section 5.4, against the coarsest colouring
    (Algorithm 1 in core).  Prints one JSON line with a row per run."""
    import numpy as np
    import torch
    import paper_2607_02603_amd as wl
    from paper_2607_02603_amd import inputs
    dev = torch.device("cuda:0")
    gens = {
        "rmat20": lambda: inputs.rmat(20, 16),
        "rmat20dir": lambda: inputs.rmat(20, 16, directed=True),
        "chunglu1m": lambda: inputs.chung_lu(1_000_000, 16_000_000),
        "rmat22": lambda: inputs.rmat(22, 16),
    }
    rows = []
    for name, gen in gens.items():
        t0 = time.perf_counter()
        g = gen()
        rp = np.asarray(g.row_ptr, np.uint64)
        hg = wl.Graph.from_numpy(g.n, rp, g.col, None, device=None)
        hg = wl.Graph(g.n, hg.row_ptr.pin_memory(), hg.col_idx.pin_memory(), None)
        dg = wl.Graph.from_numpy(g.n, rp, g.col, None, device=dev)
        log(f"{name}: n={g.n} nnz={g.nnz} built in {time.perf_counter() - t0:.1f}s")
        _, k_star, r_star = wl.wl_stable_coloring(dg, None, 0)
        torch.cuda.synchronize()
        del dg
        for nb in (1, 2, 4):
            mb = -(-g.nnz // nb)
            for mode, opt in (("fixed point", 0), ("early stop", wl.WL_BATCHED_EARLY_STOP)):
                if nb == 1 and opt:
                    continue
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                _, k, r, outer, coarsest = wl.wl_stable_coloring_batched(hg, None, 0, mb,
                                                                         options=opt)
                torch.cuda.synchronize()
                dt = time.perf_counter() - t1
                row = {"graph": STUDY_GRAPHS[name], "n": g.n, "nnz": g.nnz, "N_b": nb,
                       "M_b": mb, "outer_loop": mode, "colours": k,
                       "colours_pct_of_n": 100.0 * k / g.n,
                       "coarsest_colours": k_star,
                       "excess_pct_over_coarsest": 100.0 * (k - k_star) / k_star,
                       "outer_iterations": outer, "rounds": r, "coarsest": coarsest,
                       "seconds": dt}
                rows.append(row)
                log(f"  N_b={nb} {mode:11s}: colours {k} ({row['colours_pct_of_n']:.2f}% of n,"
                    f" +{row['excess_pct_over_coarsest']:.3f}% over {k_star}), outer {outer},"
                    f" coarsest {coarsest}, {dt:.2f}s")
        del hg, g
    print(json.dumps({"study": "reduction quality of Algorithm 2 on synthetic graphs",
                      "arithmetic": ARITH[args.arith][1], "seed": 0, "rows": rows}),
          flush=True)


def oracle_timing(args):
    """The CPU oracle on the configurations it finishes in minutes, on this
    host's cores: Algorithm 1 (oracle (a)), classic refinement (oracle (b))
    and splitter-based refinement (oracle (b'), one thread, no rounds) to
    the stable colouring, whole runs, timed around the call.  The thread
    count is OMP_NUM_THREADS (the oracle's images are OpenMP loops; its
    sorts run on one thread).  One JSON line per run."""
    if args.oracle_threads:
        os.environ["OMP_NUM_THREADS"] = str(args.oracle_threads)
    import oracle
    from paper_2607_02603_amd import inputs
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    cfgs = [("C1 ER n=20000 m=80000", inputs.er_graph, ("a", "b", "b'")),
            ("C2 grid 1024x1024", lambda: inputs.grid_graph(1024), ("a", "b", "b'")),
            ("C3 Chung-Lu n=4e6", inputs.chung_lu, ("a", "b'"))]
    for name, gen, which in cfgs:
        g = gen()
        for w in which:
            f = {"a": oracle.stable_coloring, "b": oracle.classic_coloring,
                 "b'": oracle.splitter_coloring}[w]
            t0 = time.perf_counter()
            r = f(g.row_ptr, g.col)
            dt = time.perf_counter() - t0
            rec = {"oracle": w, "config": name, "n": g.n, "nnz": g.nnz, "colours": r[1],
                   "seconds": dt, "threads": 1 if w == "b'" else threads}
            if w == "b'":
                rec["splitter_visits"] = r[2]
            else:
                rec["rounds"] = r[2]
            print(json.dumps(rec), flush=True)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def make_graph(name, device):
    import torch
    from paper_2607_02603_amd import inputs
    import paper_2607_02603_amd as wl
    if name == "er":
        g = inputs.er_graph()
    elif name == "grid":
        g = inputs.grid_graph(1024)
    elif name == "chunglu":
        g = inputs.chung_lu(device=device)
    elif name == "rmat27":
        g = inputs.rmat(27, 16, device=device)
    else:
        raise SystemExit(f"unknown workload {name}")
    if isinstance(g.row_ptr, torch.Tensor):
        rp = g.row_ptr
        if g.nnz < 2**31 and name != "rmat27":
            rp = rp.to(torch.int32)
        return wl.Graph(g.n, rp, g.col, symmetric=True), g
    return wl.Graph.from_numpy(g.n, g.row_ptr, g.col, device=device, symmetric=True), g


KINDS = ("gather", "pb", "uniform")
KIND_KERNELS = {
    "pb": "k_pb_scatter1+k_pb_scatter2+k_pb_accum (propagation-blocking image, one launch "
          "= its three passes)",
    "gather": "k_spmv_q+k_spmv_mid (gathering image of the live rows)",
    "uniform": "k_deg_hist (one-colour round)",
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pb_image_rmat27_traffic.json")
CALL_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "call_rmat27_traffic.json")
GOLDEN_DIR = os.path.join(ROOT, "tests", "golden")


def image_roofline(work, kind_ms, rp_bytes, workload, arith="fp"):
    """Roofline of the dominant image kind (largest device time per step):
    algorithmic bytes per launch (12 B per entry read: 4 B column index and
    the 8 B value of its colour; per row the row pointer and the 8 B image)
    over its average launch time from the library's HIP events."""
    ms = {kd: sum(m[kd] for m in kind_ms) / len(kind_ms) for kd in KINDS}
    kd = max(KINDS, key=lambda x: ms[x])
    w = work[kd]
    launches = max(1, w["launches"])
    bytes_per_launch = (12 * w["entries"] + (rp_bytes + 8) * w["rows"]) / launches
    avg_s = ms[kd] / 1e3 / launches
    achieved = bytes_per_launch / avg_s / 1e9 if avg_s > 0 else 0.0
    traffic = None
    if kd == "pb" and workload == "rmat27" and arith == "fp" and os.path.exists(TRAFFIC_FILE):
        from paper_2607_02603_amd import profsum
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        if t.get("source_sha256") == profsum.source_hash():
            traffic = t["traffic_bytes_per_launch"]
    return {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "kernel": KIND_KERNELS[kd],
            "launches_per_step": launches, "avg_launch_ms": avg_s * 1e3,
            "bytes_per_launch": bytes_per_launch}


def call_traffic(workload, arith, call_ms):
    """Measured HBM traffic of the whole call: the counter bytes of every
    library kernel of one call (profiles/call_rmat27_traffic.json, taken by
    rocprofv3 on the same workload) over that call's summed kernel time, and
    over this run's device time of the call.  None when the profile was taken
    on other kernel sources."""
    if workload != "rmat27" or arith != "fp" or not os.path.exists(CALL_TRAFFIC_FILE):
        return None
    from paper_2607_02603_amd import profsum
    with open(CALL_TRAFFIC_FILE) as f:
        t = json.load(f)
    if t.get("sources_sha256") != profsum.sources_hash():
        return None
    return {"bytes": t["bytes"], "profiled_kernel_ms": t["kernel_ms"],
            "frac_of_kernel_time": t["frac_of_8tbs"],
            "frac_of_call_time": t["bytes"] / (call_ms / 1e3) / (HBM_PEAK_GBS * 1e9),
            "source": os.path.relpath(CALL_TRAFFIC_FILE, ROOT)}


def golden_check(workload, arith, colors, k, rounds):
    """SHA-256 of the colour array against the oracle's stored result for
    this workload (tests/golden, written from oracle/ only), or None."""
    import hashlib
    import numpy as np
    name = {("rmat27", "fp"): "rmat27", ("rmat27", "ring64"): "rmat27_ring64",
            ("chunglu", "fp"): "chunglu"}.get((workload, arith))
    path = os.path.join(GOLDEN_DIR, f"full_{name}.json") if name else None
    if not path or not os.path.exists(path):
        return None
    with open(path) as f:
        gold = json.load(f)
    host = colors.cpu().numpy().view(np.uint32)
    sha = hashlib.sha256(host.astype("<u4").tobytes()).hexdigest()
    return {"golden": os.path.relpath(path, ROOT),
            "equal_to_oracle": sha == gold["sha256"] and (k, rounds) == (gold["colours"],
                                                                         gold["rounds"])}


def cpu_baseline(dg, seconds_target=15.0, q=0):
    """The CPU oracle (one randomized round: image + relabel) on a bounded
    sample of the same graph: the first rows of the CSR, with a pseudo-random
    colouring of 2^20 colours.  Returns the sample's per-round rate in GTEPS
    (entries of the sample over the time of that one round): a rate per
    round, not a time to the stable colouring."""
    import numpy as np
    import oracle
    rp = dg.row_ptr.cpu().numpy().astype(np.uint64)
    n = dg.n
    # grow the sample until the oracle takes a few seconds, then extrapolate
    rows = min(n, 1 << 16)
    rng = np.random.default_rng(0)
    colors = rng.integers(0, 1 << 20, size=n, dtype=np.uint32)
    best = None
    while True:
        m_s = int(rp[rows])
        col = dg.col_idx[:m_s].cpu().numpy().view(np.uint32)
        sub_rp = rp[: rows + 1].copy()
        t0 = time.perf_counter()
        z = oracle.image(sub_rp, col, None, colors, 1 << 20, 0, 1, q)
        oracle.relabel(colors[:rows], z)
        dt = time.perf_counter() - t0
        best = (rows, m_s, dt)
        if dt > seconds_target / 3 or rows == n:
            break
        rows = min(n, rows * 4)
    rows, m_s, dt = best
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": m_s / dt / 1e9, "unit": "GTEPS", "cores": threads,
            "kind": "oracle",
            "sample": f"one oracle round over the first {rows} rows ({m_s} entries) of the "
                      f"same graph with 2^20 pseudo-random colours, {dt:.2f} s: the image on "
                      f"{threads} threads (OpenMP), the relabel (qsort) on 1 thread; a per-round "
                      f"rate (entries / round time), not a time-to-stable"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="rmat27", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--arith", default="fp", choices=sorted(ARITH),
                    help="arithmetic of the image step: F_p (default) or Z/2^64")
    ap.add_argument("--batched-mode", default="streamed", choices=sorted(BATCHED_MODES),
                    help="how the out-of-core workload (rmat28b) is refined")
    ap.add_argument("--verify", action="store_true",
                    help="rmat28b: also run the in-core colouring and compare")
    ap.add_argument("--study", choices=["reduction"],
                    help="instead of the benchmark: the reduction-quality study of "
                         "Algorithm 2 (N_b = 1, 2, 4) on synthetic graphs")
    ap.add_argument("--oracle-timing", action="store_true",
                    help="instead of the benchmark: time the CPU oracles on C1-C3")
    ap.add_argument("--oracle-threads", type=int, default=0,
                    help="--oracle-timing: OMP_NUM_THREADS for the oracle (0: as set)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first copy 1 GiB device-to-device (a plain copy kernel of "
                         "known size, to calibrate rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.oracle_timing:
        return oracle_timing(args)
    import paper_2607_02603_amd as wl
    wl.wl_set_precision(ARITH[args.arith][0])
    if args.study == "reduction":
        return study_reduction(args)
    if args.workload in ("rmat28b", "rmat29s"):
        return bench_batched(args)
    import torch
    dev = torch.device("cuda:0")
    if args.copy_probe:
        src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    t0 = time.perf_counter()
    dg, _ = make_graph(args.workload, dev)
    torch.cuda.synchronize()
    log(f"graph {args.workload}: n={dg.n} nnz={dg.nnz} built in "
        f"{time.perf_counter() - t0:.1f}s")
    ws = wl.workspace(wl.wl_workspace_size(dg), dev)
    colors = torch.empty(dg.n, dtype=torch.int32, device=dev)
    for i in range(args.warmup):
        _, k, rounds = wl.wl_stable_coloring(dg, None, 0, 0, colors, ws)
        log(f"warmup {i}: colours={k} rounds={rounds}")
    # untimed run: work of every image launch (rows, entries read)
    wl.wl_stats_enable(wl.WL_STATS_TIME | wl.WL_STATS_WORK)
    _, k0, r0 = wl.wl_stable_coloring(dg, None, 0, 0, colors, ws)
    work = wl.wl_stats_get()
    check = golden_check(args.workload, args.arith, colors, k0, r0)
    log(f"result against the oracle's stored colouring: {check}")
    # timed runs: HIP events around every image launch on the library's stream
    wl.wl_stats_enable(wl.WL_STATS_TIME)
    torch.cuda.synchronize()
    times, kind_ms, call_ms = [], [], []
    for i in range(args.steps):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        _, k, rounds = wl.wl_stable_coloring(dg, None, 0, 0, colors, ws)
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t1)
        st = wl.wl_stats_get()
        kind_ms.append({kd: st[kd]["ms"] for kd in KINDS})
        call_ms.append(st["call_ms"])
        log(f"step {i}: {times[-1] * 1e3:.2f} ms colours={k} rounds={rounds} image ms: "
            + ", ".join(f"{kd} {st[kd]['ms']:.2f} ({st[kd]['launches']})" for kd in KINDS))
    wl.wl_stats_enable(0)
    # the same calls without the per-launch events: each event record is one
    # more queue packet (a few microseconds), which shows on workloads with
    # hundreds of rounds
    plain = []
    for i in range(args.steps):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        wl.wl_stable_coloring(dg, None, 0, 0, colors, ws)
        torch.cuda.synchronize()
        plain.append(time.perf_counter() - t1)
    log(f"without image timing events: {sum(plain) / len(plain) * 1e3:.2f} ms per call")
    step_s = sum(times) / len(times)
    gteps = dg.nnz * rounds / step_s / 1e9
    rp_bytes = 8 if dg.row_ptr.dtype == torch.int64 else 4
    roofline = image_roofline(work, kind_ms, rp_bytes, args.workload, args.arith)
    # CSR entries the image launches actually read (rows of classes that
    # cannot split are skipped)
    active = sum(work[kd]["entries"] for kd in KINDS)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(dg, q=ARITH[args.arith][0])
        log(f"cpu baseline: {cpu}")
    out = {
        "metric": "GTEPS per refinement round (directed CSR entries x rounds / "
                  "time-to-stable-coloring)",
        "value": gteps,
        "unit": "GTEPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload]["desc"], "n": dg.n,
                   "arithmetic": ARITH[args.arith][1],
                   "nnz": dg.nnz, "colours": k, "rounds": rounds,
                   "time_to_stable_ms": step_s * 1e3,
                   "time_to_stable_ms_without_image_events": sum(plain) / len(plain) * 1e3,
                   "image_ms_per_step": {kd: sum(m[kd] for m in kind_ms) / len(kind_ms)
                                         for kd in KINDS},
                   "active_entries_per_step": active,
                   "active_edge_gteps": active / step_s / 1e9,
                   "call_traffic": call_traffic(args.workload, args.arith,
                                                sum(call_ms) / len(call_ms)),
                   "check": check},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
