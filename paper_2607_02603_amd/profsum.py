"""Summaries of rocprofv3 output (SQLite databases) for the files under
profiles/.

    python -m paper_2607_02603_amd.profsum trace DB CALLS TITLE COMMAND > out.md
    python -m paper_2607_02603_amd.profsum traffic FETCH_DB WRITE_DB KERNELS... > out.json
    python -m paper_2607_02603_amd.profsum counters KERNELS -- DB... > out.md
    python -m paper_2607_02603_amd.profsum calltraffic FETCH_DB WRITE_DB TRACE_DB CALLS > out.json
    python -m paper_2607_02603_amd.profsum dispatches DB TITLE COMMAND > out.md
    python -m paper_2607_02603_amd.profsum reqsizes REQ_DB FETCH_DB TITLE COMMAND > out.md
    python -m paper_2607_02603_amd.profsum bandwidth REQ_DB WRITE_DB TRACE_DB TITLE COMMAND > out.md

'trace' tabulates the library's kernels of a --kernel-trace run (per-call
figures are totals divided by CALLS, the number of library calls the traced
program made).  'traffic' sums, per launch of the propagation-blocking image
(the kernels named, matched by prefix), the FETCH_SIZE and WRITE_SIZE
counters of two --pmc runs and scales them by what the same counters read for
the 1 GiB device-to-device copy that bench.py --copy-probe issues first
(bytes moved / counter value); the result records the SHA-256 of the source
file of those kernels so that a stale figure is not reported.  'counters'
tabulates, per kernel of the last library call (names matched by prefix,
comma-separated), every counter of one or more --pmc databases (one per
counter pass), summed over the kernel's dispatches and hardware instances,
with the ratios that name a kernel's bound.  'calltraffic' gives the HBM
bytes of every library kernel of one call (the last call of the two --pmc
runs, calibrated like 'traffic') and the call's summed kernel time (from a
--kernel-trace run making CALLS library calls), with the SHA-256 of all the
library's kernel sources.  'dispatches' lists, for the last library call
of a --kernel-trace run, every dispatch's duration per kernel in launch
order.  'reqsizes' checks the copy calibration of FETCH_SIZE per kernel: from
a --pmc run of TCC_EA0_RDREQ and its 32-, 64- and 128-byte parts, the read
bytes 32 R32 + 64 R64 + 128 R128 of every library kernel of the last call
(and of the copy, which must come out at 1 GiB), beside FETCH_SIZE scaled by
the copy factor.  FETCH_SIZE's formula takes 128-byte requests from
TCC_BUBBLE; where that does not count them, a 128-byte read counts as 64
bytes, so the copy factor is right for kernels that read whole 128-byte lines
and too large for kernels whose reads are 32 or 64 bytes.  'bandwidth' lists
every library kernel of the last call with its summed duration (from a
--kernel-trace run), its read bytes by request size and its WRITE_SIZE bytes
(scaled by the copy's factor), and the rate they give.
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


def sources_hash():
    """SHA-256 over the library's sources (csrc/, sorted by name)."""
    h = hashlib.sha256()
    d = os.path.join(_HERE, "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".h", ".hip")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


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



def _last_call(ev):
    lib = [(n, c) for n, c in ev if _is_lib(n)]
    starts = [i for i, (n, _) in enumerate(lib) if "k_iota_zero" in n]
    return lib[starts[-1]:] if starts else lib


def counters(kernels, dbs):
    """{kernel: {counter: value summed over its dispatches}} over the last
    library call of each database (one database per counter pass)."""
    out = {k: {"dispatches": 0} for k in kernels}
    npass = {k: {} for k in kernels}  # passes that collected each counter
    for db in dbs:
        seen = {k: 0 for k in kernels}
        got = {k: {} for k in kernels}
        for n, c in _last_call(_pmc(db)):
            s = _short(n)
            for k in kernels:
                if s.startswith(k):
                    seen[k] += 1
                    for cn, v in c.items():
                        got[k][cn] = got[k].get(cn, 0.0) + v
        for k in kernels:
            out[k]["dispatches"] = max(out[k]["dispatches"], seen[k])
            for cn, v in got[k].items():
                out[k][cn] = out[k].get(cn, 0.0) + v
                npass[k][cn] = npass[k].get(cn, 0) + 1
    # a counter collected in several passes (GRBM_GUI_ACTIVE): their mean
    for k in kernels:
        for cn, m in npass[k].items():
            out[k][cn] /= m
    return out


def counters_markdown(kernels, dbs, cu_num=256):
    res = counters(kernels, dbs)
    names = sorted({cn for k in kernels for cn in res[k] if cn != "dispatches"})
    out = ["| counter | " + " | ".join(kernels) + " |",
           "|---|" + "---|" * len(kernels)]
    for cn in ["dispatches"] + names:
        out.append(f"| {cn} | " + " | ".join(f"{res[k].get(cn, float('nan')):.4g}"
                                            for k in kernels) + " |")
    # ratios used to name each kernel's bound
    def row(label, f):
        vals = []
        for k in kernels:
            try:
                vals.append(f"{f(res[k]):.3g}")
            except (KeyError, ZeroDivisionError):
                vals.append("n/a")
        out.append(f"| {label} | " + " | ".join(vals) + " |")
    out += ["", "| derived | " + " | ".join(kernels) + " |", "|---|" + "---|" * len(kernels)]
    # GRBM_GUI_ACTIVE is summed over the 8 XCDs: per XCD it is the
    # dispatch's busy cycles
    gui = lambda r: r["GRBM_GUI_ACTIVE"] / 8  # noqa: E731
    row("busy cycles per dispatch (GRBM_GUI_ACTIVE / 8 / dispatches)",
        lambda r: gui(r) / r["dispatches"])
    row("mean waves per CU (4 x SQ_WAVE_CYCLES / busy cycles / CUs; 32 max)",
        lambda r: 4 * r["SQ_WAVE_CYCLES"] / gui(r) / cu_num)
    row("VALU busy, % (SQ_ACTIVE_INST_VALU / CUs / busy cycles)",
        lambda r: 100 * r["SQ_ACTIVE_INST_VALU"] / cu_num / gui(r))
    row("LDS busy, % (SQ_LDS_IDX_ACTIVE / CUs / busy cycles)",
        lambda r: 100 * r["SQ_LDS_IDX_ACTIVE"] / cu_num / gui(r))
    row("LDS bank-conflict stalls, % (SQ_LDS_BANK_CONFLICT / CUs / busy cycles)",
        lambda r: 100 * r["SQ_LDS_BANK_CONFLICT"] / cu_num / gui(r))
    row("LDS bank conflicts per LDS busy cycle",
        lambda r: r["SQ_LDS_BANK_CONFLICT"] / r["SQ_LDS_IDX_ACTIVE"])
    row("wave-cycles waiting on LDS / wave-cycles (SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES)",
        lambda r: r["SQ_WAIT_INST_LDS"] / r["SQ_WAVE_CYCLES"])
    row("wave-cycles waiting on anything / wave-cycles (SQ_WAIT_ANY / SQ_WAVE_CYCLES)",
        lambda r: r["SQ_WAIT_ANY"] / r["SQ_WAVE_CYCLES"])
    row("LDS instructions per wave", lambda r: r["SQ_INSTS_LDS"] / r["SQ_WAVES"])
    row("LDS atomic instructions per wave", lambda r: r["SQ_INSTS_LDS_ATOMIC"] / r["SQ_WAVES"])
    row("VALU instructions per wave", lambda r: r["SQ_INSTS_VALU"] / r["SQ_WAVES"])
    row("vector memory reads per wave",
        lambda r: r["SQ_INSTS_VMEM_RD"] / r["SQ_WAVES"])
    row("vector memory writes per wave", lambda r: r["SQ_INSTS_VMEM_WR"] / r["SQ_WAVES"])
    row("memory writes of 64 B, % of write requests (TCC_EA0_WRREQ_64B / TCC_EA0_WRREQ)",
        lambda r: 100 * r["TCC_EA0_WRREQ_64B"] / r["TCC_EA0_WRREQ"])
    row("memory reads of 32 B, % of read requests (TCC_EA0_RDREQ_32B / TCC_EA0_RDREQ)",
        lambda r: 100 * r["TCC_EA0_RDREQ_32B"] / r["TCC_EA0_RDREQ"])
    return "\n".join(out)


def call_traffic(fetch_db, write_db, trace_db, calls):
    t = traffic(fetch_db, write_db, [])
    _, kernel_ms = trace_table(trace_db, calls)
    b = t["call"]["bytes"]
    return {"what": "HBM bytes (FETCH_SIZE + WRITE_SIZE, calibrated on a 1 GiB copy) of every "
                    "library kernel of one stable colouring, and the summed duration of those "
                    "kernels",
            "sources_sha256": sources_hash(), "bytes": b, "kernel_ms": kernel_ms,
            "tb_per_s": b / (kernel_ms / 1e3) / 1e12,
            "frac_of_8tbs": b / (kernel_ms / 1e3) / 8e12,
            "fetch_scale": t["fetch"]["scale"], "write_scale": t["write"]["scale"],
            "top_kernels_bytes": t["call"]["top_kernels_bytes"]}

def dispatches_markdown(db, title, command, top=20):
    cur = sqlite3.connect(db).cursor()
    cols = [r[1] for r in cur.execute("pragma table_info(kernels)")]
    ki = cols.index("kernel_name") if "kernel_name" in cols else cols.index("name")
    st, en = cols.index("start"), cols.index("end")
    rows = [r for r in cur.execute("select * from kernels order by start").fetchall()
            if _is_lib(r[ki])]
    starts = [i for i, r in enumerate(rows) if "k_iota_zero" in r[ki]]
    rows = rows[starts[-1]:] if starts else rows
    per = {}
    for r in rows:
        per.setdefault(_short(r[ki]), []).append((r[en] - r[st]) / 1e6)
    total = sum(sum(v) for v in per.values())
    span = (rows[-1][en] - rows[0][st]) / 1e6 if rows else 0.0
    out = [f"# {title}", "", "Command (repository root, on the MI355X machine):", "",
           f"    {command}", "",
           "The last library call of the trace; library kernels, ms per dispatch in launch "
           f"order ({top} kernels of largest total).  Kernel time of the call: {total:.2f} ms; "
           f"first start to last end: {span:.2f} ms.", "",
           "| kernel | dispatches | ms per dispatch, in order | total ms |", "|---|---|---|---|"]
    for name, v in sorted(per.items(), key=lambda kv: -sum(kv[1]))[:top]:
        out.append(f"| {name} | {len(v)} | " + ", ".join(f"{x:.3f}" for x in v) +
                   f" | {sum(v):.3f} |")
    return "\n".join(out)


_REQ = ("TCC_EA0_RDREQ", "TCC_EA0_RDREQ_32B", "TCC_EA0_RDREQ_64B", "TCC_EA0_RDREQ_128B")


def _req_bytes(c):
    return 32.0 * c["TCC_EA0_RDREQ_32B"] + 64.0 * c["TCC_EA0_RDREQ_64B"] + \
        128.0 * c["TCC_EA0_RDREQ_128B"]


def reqsizes(req_db, fetch_db):
    """Per kernel of the last library call: read requests by size, the read
    bytes they give, and FETCH_SIZE scaled by the copy factor."""
    ev_r, ev_f = _pmc(req_db), _pmc(fetch_db)
    copy_r = [c for n, c in ev_r if "copyBuffer" in n and all(k in c for k in _REQ)]
    copy_f = [c["FETCH_SIZE"] for n, c in ev_f if "copyBuffer" in n and "FETCH_SIZE" in c]
    if not copy_r or not copy_f:
        raise SystemExit("no copy-kernel dispatch in the request or FETCH_SIZE run")
    scale = (1 << 30) / (copy_f[0] * 1024.0)
    per = {}
    for n, c in _last_call(ev_r):
        e = per.setdefault(_short(n), {k: 0.0 for k in _REQ})
        for k in _REQ:
            e[k] += c.get(k, 0.0)
    fetch = {}
    for n, c in _last_call(ev_f):
        fetch[_short(n)] = fetch.get(_short(n), 0.0) + c.get("FETCH_SIZE", 0.0) * 1024.0 * scale
    rows = []
    for name, e in per.items():
        rows.append({"kernel": name, **{k: e[k] for k in _REQ}, "bytes": _req_bytes(e),
                     "fetch_scaled": fetch.get(name, 0.0),
                     "unsized": e["TCC_EA0_RDREQ"] - e["TCC_EA0_RDREQ_32B"] -
                     e["TCC_EA0_RDREQ_64B"] - e["TCC_EA0_RDREQ_128B"]})
    rows.sort(key=lambda r: -r["fetch_scaled"])
    c0 = copy_r[0]
    return {"copy": {"bytes": _req_bytes(c0), "expected": float(1 << 30),
                     **{k: c0[k] for k in _REQ}, "fetch_kib": copy_f[0], "fetch_scale": scale},
            "kernels": rows,
            "total_bytes": sum(r["bytes"] for r in rows),
            "total_fetch_scaled": sum(r["fetch_scaled"] for r in rows)}


def reqsizes_markdown(req_db, fetch_db, title, command, top=20):
    r = reqsizes(req_db, fetch_db)
    c = r["copy"]
    out = [f"# {title}", "", "Commands (repository root, on the MI355X machine):", ""]
    out += [f"    {x}" for x in command.split(" ;; ")]
    out += ["",
            f"The 1 GiB copy that `--copy-probe` issues first: {c['TCC_EA0_RDREQ_128B']:,.0f} "
            f"128-byte, {c['TCC_EA0_RDREQ_64B']:,.0f} 64-byte and {c['TCC_EA0_RDREQ_32B']:,.0f} "
            f"32-byte read requests, {c['bytes'] / (1 << 30):.4f} GiB by request size; "
            f"FETCH_SIZE reads {c['fetch_kib']:,.0f} KiB, a factor of {c['fetch_scale']:.3f}.",
            "",
            "Library kernels of the last call, by scaled FETCH_SIZE (GB = 1e9 bytes; "
            "`by size` = 32 R32 + 64 R64 + 128 R128):", "",
            "| kernel | R32 | R64 | R128 | read GB by size | FETCH_SIZE x factor, GB | ratio |",
            "|---|---|---|---|---|---|---|"]
    for k in r["kernels"][:top]:
        ratio = k["fetch_scaled"] / k["bytes"] if k["bytes"] else float("nan")
        out.append(f"| {k['kernel']} | {k['TCC_EA0_RDREQ_32B']:,.0f} | "
                   f"{k['TCC_EA0_RDREQ_64B']:,.0f} | {k['TCC_EA0_RDREQ_128B']:,.0f} | "
                   f"{k['bytes'] / 1e9:.3f} | {k['fetch_scaled'] / 1e9:.3f} | {ratio:.2f} |")
    unsized = sum(k["unsized"] for k in r["kernels"])
    out += ["", f"All library kernels of the call: {r['total_bytes'] / 1e9:.2f} GB read by "
            f"request size against {r['total_fetch_scaled'] / 1e9:.2f} GB of scaled FETCH_SIZE; "
            f"read requests outside the three sizes: {unsized:,.0f}."]
    return "\n".join(out)


def _trace_last_call(db):
    """{kernel: (dispatches, ms)} over the last library call of a trace."""
    cur = sqlite3.connect(db).cursor()
    cols = [r[1] for r in cur.execute("pragma table_info(kernels)")]
    ki = cols.index("kernel_name") if "kernel_name" in cols else cols.index("name")
    st, en = cols.index("start"), cols.index("end")
    rows = [r for r in cur.execute("select * from kernels order by start").fetchall()
            if _is_lib(r[ki])]
    starts = [i for i, r in enumerate(rows) if "k_iota_zero" in r[ki]]
    rows = rows[starts[-1]:] if starts else rows
    out = {}
    for r in rows:
        d, ms = out.get(_short(r[ki]), (0, 0.0))
        out[_short(r[ki])] = (d + 1, ms + (r[en] - r[st]) / 1e6)
    return out


def bandwidth(req_db, write_db, trace_db):
    ev_r, ev_w = _pmc(req_db), _pmc(write_db)
    copy_w = [c["WRITE_SIZE"] for n, c in ev_w if "copyBuffer" in n and "WRITE_SIZE" in c]
    if not copy_w:
        raise SystemExit(f"{write_db}: no copy-kernel dispatch to calibrate WRITE_SIZE")
    wscale = (1 << 30) / (copy_w[0] * 1024.0)
    rd, wr = {}, {}
    for n, c in _last_call(ev_r):
        rd[_short(n)] = rd.get(_short(n), 0.0) + _req_bytes({k: c.get(k, 0.0) for k in _REQ})
    for n, c in _last_call(ev_w):
        wr[_short(n)] = wr.get(_short(n), 0.0) + c.get("WRITE_SIZE", 0.0) * 1024.0 * wscale
    tr = _trace_last_call(trace_db)
    rows = []
    for name, (d, ms) in tr.items():
        r, w = rd.get(name, 0.0), wr.get(name, 0.0)
        rows.append({"kernel": name, "dispatches": d, "ms": ms, "read": r, "write": w,
                     "tb_per_s": (r + w) / (ms / 1e3) / 1e12 if ms > 0 else 0.0})
    rows.sort(key=lambda x: -x["ms"])
    return {"write_scale": wscale, "kernels": rows}


def bandwidth_markdown(req_db, write_db, trace_db, title, command, top=25):
    b = bandwidth(req_db, write_db, trace_db)
    out = [f"# {title}", "", "Commands (repository root, on the MI355X machine):", ""]
    out += [f"    {x}" for x in command.split(" ;; ")]
    out += ["", "Library kernels of the last call by duration: read bytes by request size "
            "(32 R32 + 64 R64 + 128 R128), WRITE_SIZE scaled by the 1 GiB copy "
            f"(x {b['write_scale']:.3f}); GB = 1e9 bytes; the rate is (read + write) / duration "
            "against 8 TB/s.", "",
            "| kernel | dispatches | ms | read GB | write GB | TB/s | % of 8 TB/s |",
            "|---|---|---|---|---|---|---|"]
    for k in b["kernels"][:top]:
        out.append(f"| {k['kernel']} | {k['dispatches']} | {k['ms']:.3f} | {k['read'] / 1e9:.3f} | "
                   f"{k['write'] / 1e9:.3f} | {k['tb_per_s']:.2f} | {k['tb_per_s'] / 8 * 100:.1f} |")
    return "\n".join(out)


def main(argv):
    if len(argv) >= 5 and argv[0] == "trace":
        print(trace_markdown(argv[1], int(argv[2]), argv[3], argv[4]))
    elif len(argv) >= 4 and argv[0] == "counters" and "--" in argv:
        cut = argv.index("--")
        print(counters_markdown(argv[1].split(","), argv[cut + 1:]))
    elif len(argv) == 5 and argv[0] == "calltraffic":
        print(json.dumps(call_traffic(argv[1], argv[2], argv[3], int(argv[4])), indent=1))
    elif len(argv) == 4 and argv[0] == "dispatches":
        print(dispatches_markdown(argv[1], argv[2], argv[3]))
    elif len(argv) == 6 and argv[0] == "bandwidth":
        print(bandwidth_markdown(argv[1], argv[2], argv[3], argv[4], argv[5]))
    elif len(argv) == 5 and argv[0] == "reqsizes":
        print(reqsizes_markdown(argv[1], argv[2], argv[3], argv[4]))
    elif len(argv) >= 4 and argv[0] == "traffic":
        print(json.dumps(traffic(argv[1], argv[2], argv[3:]), indent=1))
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
