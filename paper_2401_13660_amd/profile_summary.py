"""Summaries of rocprofv3 result databases, for the figures kept under profiles/.

    python -m paper_2401_13660_amd.profile_summary trace DB [--last N]
        per kernel: calls, total and average duration, and the average of the
        last N dispatches (the timed launches of a bench run).

    python -m paper_2401_13660_amd.profile_summary traffic --workload NAME --kernel SUBSTR
            --fetch DB --write DB --copy-fetch DB --copy-write DB --copy-mib MIB [--out FILE]
        HBM bytes per launch of the matching kernel from one FETCH_SIZE and one
        WRITE_SIZE pass (KiB per dispatch), each scaled by the ratio of true bytes
        to what the same counter reads for a plain device copy of MIB MiB; the
        record is merged into FILE (profiles/traffic.json by default) together
        with the digest of the kernel's sources, so that a later change of the
        kernel invalidates it.

The databases are the ``*_results.db`` files that ``rocprofv3 -d DIR -o run``
writes; only the ``kernels`` and ``counters_collection`` views are read.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sqlite3
from collections import defaultdict

_PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(_PKG)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")

# The files that define the forward scan kernels (plain and time-split) and their
# launch configuration, and
# those of the convolution kernel (its launch lives in mbscan.hip's conv_fwd_k).
KERNEL_SOURCES = ("scan_tiled.hpp", "scan_ts2.hpp", "device_math.hpp", "scan_params.hpp")
CONV_KERNEL_SOURCES = ("conv1d.hpp", "device_math.hpp")


def kernel_sources_digest(sources=KERNEL_SOURCES) -> str:
    h = hashlib.sha256()
    for name in sources:
        with open(os.path.join(_PKG, "csrc", name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def dispatches(db: str):
    """[(kernel name, duration ns)] in dispatch order."""
    con = sqlite3.connect(db)
    try:
        rows = con.execute("select name, start, end from kernels order by start").fetchall()
    finally:
        con.close()
    return [(n, e - s) for n, s, e in rows]


def trace_table(db: str, last: int = 0):
    per = defaultdict(list)
    for name, dur in dispatches(db):
        per[name].append(dur)
    out = []
    for name, durs in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        row = {"kernel": name, "calls": len(durs), "total_us": sum(durs) / 1e3,
               "avg_us": sum(durs) / len(durs) / 1e3, "min_us": min(durs) / 1e3}
        if last and len(durs) >= last:
            row[f"avg_last{last}_us"] = sum(durs[-last:]) / last / 1e3
        out.append(row)
    return out


def counter_per_dispatch(db: str, counter: str, kernel_substr: str) -> float:
    """Mean over the matching dispatches of the counter's per-dispatch value."""
    con = sqlite3.connect(db)
    try:
        rows = con.execute("select kernel_name, counter_name, value, dispatch_id from counters_collection"
                           ).fetchall()
    finally:
        con.close()
    per_dispatch = defaultdict(float)
    for kname, cname, value, did in rows:
        if kernel_substr in kname and cname == counter:
            per_dispatch[did] += value
    if not per_dispatch:
        raise SystemExit(f"no {counter} values for kernels matching {kernel_substr!r} in {db}")
    return sum(per_dispatch.values()) / len(per_dispatch)


def traffic_record(args) -> dict:
    fetch = counter_per_dispatch(args.fetch, "FETCH_SIZE", args.kernel)
    write = counter_per_dispatch(args.write, "WRITE_SIZE", args.kernel)
    cfetch = counter_per_dispatch(args.copy_fetch, "FETCH_SIZE", args.copy_kernel)
    cwrite = counter_per_dispatch(args.copy_write, "WRITE_SIZE", args.copy_kernel)
    nbytes = args.copy_mib << 20
    ffac = nbytes / (cfetch * 1024.0)
    wfac = nbytes / (cwrite * 1024.0)
    rd = fetch * 1024.0 * ffac
    wr = write * 1024.0 * wfac
    return {
        "kernel": args.kernel,
        "kernel_sources": kernel_sources_digest(CONV_KERNEL_SOURCES if args.conv else KERNEL_SOURCES),
        "fetch_size_kib_per_dispatch": round(fetch, 1),
        "write_size_kib_per_dispatch": round(write, 1),
        "copy_calibration": {"bytes": nbytes, "fetch_size_kib": round(cfetch, 1),
                             "write_size_kib": round(cwrite, 1), "fetch_factor": round(ffac, 4),
                             "write_factor": round(wfac, 4)},
        "hbm_read_bytes_per_launch": int(rd),
        "hbm_write_bytes_per_launch": int(wr),
        "hbm_bytes_per_launch": int(rd + wr),
        "commands": args.commands or [],
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("db")
    t.add_argument("--last", type=int, default=0)
    f = sub.add_parser("traffic")
    f.add_argument("--workload", required=True)
    f.add_argument("--kernel", required=True, help="substring of the kernel name")
    f.add_argument("--copy-kernel", default="copyBuffer")
    f.add_argument("--fetch", required=True)
    f.add_argument("--write", required=True)
    f.add_argument("--copy-fetch", required=True)
    f.add_argument("--copy-write", required=True)
    f.add_argument("--copy-mib", type=int, required=True)
    f.add_argument("--command", dest="commands", action="append", help="command that made a pass")
    f.add_argument("--out", default=TRAFFIC_FILE)
    f.add_argument("--conv", action="store_true", help="the record is for the convolution kernel")
    args = ap.parse_args(argv)
    if args.cmd == "trace":
        print(json.dumps(trace_table(args.db, args.last), indent=1))
        return
    rec = traffic_record(args)
    try:
        with open(args.out) as fh:
            allrec = json.load(fh)
    except (OSError, ValueError):
        allrec = {}
    allrec[args.workload] = rec
    with open(args.out, "w") as fh:
        json.dump(allrec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec, indent=1))


if __name__ == "__main__":
    main()
