"""Summaries of rocprofv3 output (SQLite databases) for the files under
profiles/.

    python -m paper_2607_02603_amd.profsum trace DB CALLS TITLE COMMAND > out.md
    python -m paper_2607_02603_amd.profsum traffic FETCH_DB WRITE_DB KERNELS... > out.json

'trace' tabulates the library's kernels of a --kernel-trace run (per-call
figures are totals divided by CALLS, the number of library calls the traced
program made).  'traffic' sums, per launch of the propagation-blocking image
(the kernels named, matched by prefix), the FETCH_SIZE and WRITE_SIZE
counters of two --pmc runs and scales them by what the same counters read for
the 1 GiB device-to-device copy that bench.py --copy-probe issues first
(bytes moved / counter value); the result records the SHA-256 of the source
file of those kernels so that a stale figure is not reported.
"""
import hashlib
import json
import os
import re
import sqlite3
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
PB_SOURCE = os.path.join(_HERE, "csrc", "wl_push.h")


def source_hash(path=PB_SOURCE):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def _short(name):
    name = name.replace("(anonymous namespace)::", "")
    return re.sub(r"\(.*", "", name).replace("void ", "").replace("wl::", "")


def _is_lib(name):
    return bool(re.search(r"wl::|\(anonymous namespace\)::k_", name)) and "Src" not in name


def trace_table(db, calls):
    cur = sqlite3.connect(db).cursor()
    cols = [r[1] for r in cur.execute("pragma table_info(kernels)")]
    ki = cols.index("kernel_name") if "kernel_name" in cols else cols.index("name")
    st, en = cols.index("start"), cols.index("end")
    agg = {}
    for r in cur.execute("select * from kernels").fetchall():
        if not _is_lib(r[ki]):
            continue
        a = agg.setdefault(_short(r[ki]), [0, 0.0])
        a[0] += 1
        a[1] += (r[en] - r[st]) / 1e6
    rows = sorted(agg.items(), key=lambda kv: -kv[1][1])
    return rows, sum(t for _, (_, t) in rows) / calls


def trace_markdown(db, calls, title, command):
    rows, per_call = trace_table(db, calls)
    out = [f"# {title}", "", "Command (repository root, on the MI355X machine):", "",
           f"    {command}", "",
           f"Library kernels only; the traced program makes {calls} library call(s): "
           f"per-call figures are totals / {calls}.", "",
           "| kernel | calls | total ms | avg ms | ms per call |", "|---|---|---|---|---|"]
    for name, (c, t) in rows:
        out.append(f"| {name} | {c} | {t:.3f} | {t / c:.4f} | {t / calls:.3f} |")
    out += ["", f"Sum of library kernel time per call: {per_call:.2f} ms."]
    return "\n".join(out)


def _pmc(db):
    cur = sqlite3.connect(db).cursor()
    rows = cur.execute("select dispatch_id, name, counter_name, counter_value "
                       "from pmc_events order by dispatch_id").fetchall()
    disp = {}
    for d, n, cn, cv in rows:
        e = disp.setdefault(d, [n, {}])
        e[1][cn] = e[1].get(cn, 0.0) + cv
    return [disp[d] for d in sorted(disp)]


def traffic(fetch_db, write_db, kernels):
    """Per-launch HBM bytes of the kernels (name prefixes) from the last
    library call in each database, scaled by the copy-kernel calibration."""
    res = {}
    for which, db, counter in (("fetch", fetch_db, "FETCH_SIZE"),
                               ("write", write_db, "WRITE_SIZE")):
        ev = _pmc(db)
        copy = [c[counter] for n, c in ev if "copyBuffer" in n and counter in c]
        if not copy:
            raise SystemExit(f"{db}: no copy-kernel dispatch to calibrate {counter}")
        scale = (1 << 30) / (copy[0] * 1024.0)  # bytes moved per counted byte
        # the last library call starts at its last k_iota_zero (or at the
        # start of the one-colour degree round)
        lib = [(n, c) for n, c in ev if _is_lib(n)]
        starts = [i for i, (n, _) in enumerate(lib) if "k_iota_zero" in n]
        lib = lib[starts[-1]:] if starts else lib
        kib = {k: 0.0 for k in kernels}
        for n, c in lib:
            s = _short(n)
            for k in kernels:
                if s.startswith(k):
                    kib[k] += c.get(counter, 0.0)
        # the whole call: every library kernel, summed per kernel name
        per = {}
        for n, c in lib:
            s = _short(n)
            per[s] = per.get(s, 0.0) + c.get(counter, 0.0) * 1024.0 * scale
        res[which] = {"counter": counter, "kib": kib, "copy_kib": copy[0], "scale": scale,
                      "bytes": sum(kib.values()) * 1024.0 * scale,
                      "call_bytes": sum(per.values()), "call_per_kernel": per}
    per_kernel = {}
    for which in ("fetch", "write"):
        for k, v in res[which].pop("call_per_kernel").items():
            per_kernel[k] = per_kernel.get(k, 0.0) + v
    top = dict(sorted(per_kernel.items(), key=lambda kv: -kv[1])[:20])
    return {"kernels": kernels, "source": os.path.relpath(PB_SOURCE, os.path.dirname(_HERE)),
            "source_sha256": source_hash(), "fetch": res["fetch"], "write": res["write"],
            "traffic_bytes_per_launch": res["fetch"]["bytes"] + res["write"]["bytes"],
            "call": {"note": "all library kernels of the last call (fetch + write, scaled "
                             "like the image's); informational, not tied to the hash above",
                     "bytes": res["fetch"]["call_bytes"] + res["write"]["call_bytes"],
                     "top_kernels_bytes": top}}


def main(argv):
    if len(argv) >= 5 and argv[0] == "trace":
        print(trace_markdown(argv[1], int(argv[2]), argv[3], argv[4]))
    elif len(argv) >= 4 and argv[0] == "traffic":
        print(json.dumps(traffic(argv[1], argv[2], argv[3:]), indent=1))
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
