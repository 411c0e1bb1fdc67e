"""The counter arithmetic of paper_2607_02603_amd.profsum on hand-made
rocprofv3 databases (a pmc_events table of dispatch, kernel name, counter and
value), so the profile summaries' figures can be checked without a GPU.

* reqsizes: read bytes are 32 R32 + 64 R64 + 128 R128; the copy of 1 GiB in
  8,388,608 128-byte requests comes out at 1 GiB, and its FETCH_SIZE of
  524,288 KiB gives the factor 2; only the last library call counts (it starts
  at its last k_iota_zero), summed per kernel name over its dispatches; a
  kernel of 64-byte reads shows FETCH_SIZE x 2 at twice its request bytes
  when FETCH_SIZE counts those 64-byte reads as 64 bytes.
* traffic: FETCH_SIZE and WRITE_SIZE scaled by the copy's factors, per
  named kernel.
* bandwidth: per kernel of the last call of a hand-made kernel trace, its
  summed duration, read bytes by request size and scaled WRITE_SIZE, and
  the rate they give.
"""
import sqlite3

import pytest

from paper_2607_02603_amd import profsum

COPY = "void __amd_rocclr_copyBuffer(...)"
IOTA = "void wl::k_iota_zero(wl::Ctx)"
EMIT = "void wl::k_live_emit<unsigned long>(wl::Ctx)"
SORT = "void wl::k_sorts<false>(wl::Ctx, int, unsigned int, unsigned int)"


def _db(path, dispatches):
    con = sqlite3.connect(path)
    con.execute("create table pmc_events (dispatch_id integer, name text, "
                "counter_name text, counter_value real)")
    for d, (name, counters) in enumerate(dispatches):
        for cn, cv in counters.items():
            # two hardware instances per counter, summed by the reader
            con.execute("insert into pmc_events values (?, ?, ?, ?)", (d, name, cn, cv / 2))
            con.execute("insert into pmc_events values (?, ?, ?, ?)", (d, name, cn, cv / 2))
    con.commit()
    con.close()
    return str(path)


def _req(r32, r64, r128):
    return {"TCC_EA0_RDREQ": r32 + r64 + r128, "TCC_EA0_RDREQ_32B": r32,
            "TCC_EA0_RDREQ_64B": r64, "TCC_EA0_RDREQ_128B": r128}


def test_reqsizes(tmp_path):
    lines = (1 << 30) // 128
    req = _db(tmp_path / "req.db", [
        (COPY, _req(0, 0, lines)),
        (IOTA, _req(0, 0, 10)),          # an earlier call: ignored
        (EMIT, _req(0, 0, 999)),
        (IOTA, _req(0, 0, 8)),           # the last call
        (EMIT, _req(0, 0, 1000)),
        (EMIT, _req(0, 0, 500)),
        (SORT, _req(4, 100, 0)),
    ])
    fetch = _db(tmp_path / "fetch.db", [
        (COPY, {"FETCH_SIZE": (1 << 30) / 2 / 1024}),
        (IOTA, {"FETCH_SIZE": 1.0}),
        (EMIT, {"FETCH_SIZE": 5.0}),
        (IOTA, {"FETCH_SIZE": 8 * 64 / 1024}),
        (EMIT, {"FETCH_SIZE": 1000 * 64 / 1024}),
        (EMIT, {"FETCH_SIZE": 500 * 64 / 1024}),
        (SORT, {"FETCH_SIZE": (4 * 32 + 100 * 64) / 1024}),
    ])
    r = profsum.reqsizes(req, fetch)
    assert r["copy"]["bytes"] == 1 << 30
    assert r["copy"]["fetch_scale"] == pytest.approx(2.0)
    k = {x["kernel"]: x for x in r["kernels"]}
    assert set(k) == {"k_iota_zero", "k_live_emit<unsigned long>", "k_sorts<false>"}
    emit = k["k_live_emit<unsigned long>"]
    assert emit["TCC_EA0_RDREQ_128B"] == 1500
    assert emit["bytes"] == 1500 * 128
    assert emit["fetch_scaled"] == pytest.approx(1500 * 128)
    srt = k["k_sorts<false>"]
    assert srt["bytes"] == 4 * 32 + 100 * 64
    assert srt["fetch_scaled"] == pytest.approx(2 * (4 * 32 + 100 * 64))
    assert srt["unsized"] == 0
    assert r["total_bytes"] == 8 * 128 + 1500 * 128 + 4 * 32 + 100 * 64
    md = profsum.reqsizes_markdown(req, fetch, "T", "cmd a ;; cmd b")
    assert "    cmd a" in md and "    cmd b" in md and "1.0000 GiB" in md


def test_traffic(tmp_path):
    fetch = _db(tmp_path / "f.db", [
        (COPY, {"FETCH_SIZE": (1 << 30) / 2 / 1024}),
        (IOTA, {"FETCH_SIZE": 1.0}),
        (EMIT, {"FETCH_SIZE": 100.0}),
    ])
    write = _db(tmp_path / "w.db", [
        (COPY, {"WRITE_SIZE": (1 << 30) / 1024}),
        (IOTA, {"WRITE_SIZE": 2.0}),
        (EMIT, {"WRITE_SIZE": 50.0}),
    ])
    t = profsum.traffic(fetch, write, ["k_live_emit"])
    assert t["fetch"]["scale"] == pytest.approx(2.0)
    assert t["write"]["scale"] == pytest.approx(1.0)
    assert t["fetch"]["bytes"] == pytest.approx(100 * 1024 * 2)
    assert t["write"]["bytes"] == pytest.approx(50 * 1024)
    assert t["traffic_bytes_per_launch"] == pytest.approx(100 * 2048 + 50 * 1024)
    assert t["call"]["bytes"] == pytest.approx((1 + 100) * 2048 + (2 + 50) * 1024)


def _trace(path, kernels):
    con = sqlite3.connect(path)
    con.execute("create table kernels (kernel_name text, start integer, end integer)")
    for name, start, end in kernels:
        con.execute("insert into kernels values (?, ?, ?)", (name, start, end))
    con.commit()
    con.close()
    return str(path)


def test_bandwidth(tmp_path):
    req = _db(tmp_path / "req.db", [
        (COPY, _req(0, 0, (1 << 30) // 128)),
        (IOTA, _req(0, 0, 1)),
        (EMIT, _req(0, 0, 1000)),
        (EMIT, _req(0, 10, 0)),
    ])
    write = _db(tmp_path / "w.db", [
        (COPY, {"WRITE_SIZE": (1 << 30) / 1024}),
        (IOTA, {"WRITE_SIZE": 1.0}),
        (EMIT, {"WRITE_SIZE": 4.0}),
        (EMIT, {"WRITE_SIZE": 6.0}),
    ])
    # times in ns; an earlier call (before the last k_iota_zero) is ignored
    tr = _trace(tmp_path / "t.db", [
        (EMIT, 0, 5_000_000),
        (IOTA, 10_000_000, 10_001_000),
        (EMIT, 10_002_000, 10_004_000),
        (EMIT, 10_005_000, 10_006_000),
    ])
    b = profsum.bandwidth(req, write, tr)
    k = {x["kernel"]: x for x in b["kernels"]}
    e = k["k_live_emit<unsigned long>"]
    assert e["dispatches"] == 2
    assert e["ms"] == pytest.approx(0.003)
    assert e["read"] == 1000 * 128 + 10 * 64
    assert e["write"] == pytest.approx(10 * 1024)
    assert e["tb_per_s"] == pytest.approx((1000 * 128 + 640 + 10240) / 3e-6 / 1e12)
    assert b["kernels"][0]["kernel"] == "k_live_emit<unsigned long>"
    md = profsum.bandwidth_markdown(req, write, tr, "T", "a ;; b")
    assert "| k_live_emit<unsigned long> | 2 | 0.003 |" in md
