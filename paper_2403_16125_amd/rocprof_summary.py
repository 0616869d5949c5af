"""Summarise a rocprofv3 results database (kernel trace and/or PMC counters).

    python -m paper_2403_16125_amd.rocprof_summary <results.db> [--kernel SUBSTR]

Prints per-kernel dispatch statistics (calls, total / average / min / max
duration in microseconds) and, when counters were collected, the per-dispatch
average of every counter per kernel.  Also usable as a library by bench.py.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import sqlite3
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)


# the sources that decide what each kernel does (device code, shared
# definitions, and the host code that prepares its launch)
KERNEL_SOURCES = {
    "estimate_kernel": ("include/arena.h", "paper_2403_16125_amd/csrc/arena_internal.h",
                        "paper_2403_16125_amd/csrc/arena_host.cpp",
                        "paper_2403_16125_amd/csrc/arena_kernels.hip"),
    "estimate_mem_kernel": ("include/arena.h", "paper_2403_16125_amd/csrc/arena_internal.h",
                            "paper_2403_16125_amd/csrc/arena_host.cpp",
                            "paper_2403_16125_amd/csrc/arena_kernels.hip"),
    "estimate_tab_kernel": ("include/arena.h", "paper_2403_16125_amd/csrc/arena_internal.h",
                            "paper_2403_16125_amd/csrc/arena_host.cpp",
                            "paper_2403_16125_amd/csrc/arena_kernels.hip"),
    "schedule_kernel": ("include/arena.h", "paper_2403_16125_amd/csrc/arena_internal.h",
                        "paper_2403_16125_amd/csrc/arena_host.cpp",
                        "paper_2403_16125_amd/csrc/arena_sched.hip"),
    "proxy_kernel": ("include/arena.h", "paper_2403_16125_amd/csrc/arena_internal.h",
                     "paper_2403_16125_amd/csrc/arena_host.cpp",
                     "paper_2403_16125_amd/csrc/arena_proxy.hip"),
}


def _code_only(text: str) -> str:
    """C/C++ source without its comments (edits to documentation do not
    change what a kernel does)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.sub(r"//[^\n]*", "", text)


def kernel_source_sha(kernel: str = "estimate_kernel") -> str:
    """Hash of the code (comments removed) of the files one kernel is built from."""
    files = [os.path.join(ROOT, f) for f in KERNEL_SOURCES[kernel]]
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def _tables(cur):
    return {r[0] for r in cur.execute("select name from sqlite_master where type in ('table','view')")}


def dispatch_stats(db: str, kernel: str | None = None):
    con = sqlite3.connect(db)
    cur = con.cursor()
    if "kernels" not in _tables(cur):
        return []
    q = ("select name, count(*), sum(duration), avg(duration), min(duration), max(duration) "
         "from kernels group by name order by sum(duration) desc")
    out = []
    for name, n, tot, avg, mn, mx in cur.execute(q):
        if kernel and kernel not in name:
            continue
        out.append(dict(name=name, calls=n, total_us=tot / 1e3, avg_us=avg / 1e3,
                        min_us=mn / 1e3, max_us=mx / 1e3))
    return out


def counter_stats(db: str, kernel: str | None = None):
    con = sqlite3.connect(db)
    cur = con.cursor()
    if "counters_collection" not in _tables(cur):
        return []
    q = ("select kernel_name, counter_name, count(distinct dispatch_id), sum(value) "
         "from counters_collection group by kernel_name, counter_name")
    out = []
    for name, counter, ndisp, total in cur.execute(q):
        if kernel and kernel not in name:
            continue
        out.append(dict(name=name, counter=counter, dispatches=ndisp,
                        per_dispatch=total / max(ndisp, 1)))
    return out


def traffic(fetch_db, write_db, copy_fetch_db, copy_write_db, kernel, copy_bytes, workload):
    """HBM bytes per launch of `kernel` from FETCH_SIZE and WRITE_SIZE runs
    (KiB per dispatch), each scaled by what the same counter reads for a plain
    elementwise copy of copy_bytes read + copy_bytes written."""
    def one(db, name, counter):
        vals = [c["per_dispatch"] for c in counter_stats(db, name) if c["counter"] == counter]
        if not vals:
            raise SystemExit(f"no {counter} for {name} in {db}")
        return max(vals)
    f_kib = one(fetch_db, kernel, "FETCH_SIZE")
    w_kib = one(write_db, kernel, "WRITE_SIZE")
    cf_kib = one(copy_fetch_db, "elementwise", "FETCH_SIZE")
    cw_kib = one(copy_write_db, "elementwise", "WRITE_SIZE")
    f_scale = copy_bytes / (cf_kib * 1024.0)
    w_scale = copy_bytes / (cw_kib * 1024.0)
    fetch_b = f_kib * 1024.0 * f_scale
    write_b = w_kib * 1024.0 * w_scale
    return dict(workload=workload, kernel=kernel, kernel_source_sha=kernel_source_sha(kernel),
                fetch_kib_per_dispatch=f_kib, write_kib_per_dispatch=w_kib,
                copy_fetch_kib=cf_kib, copy_write_kib=cw_kib, copy_bytes=copy_bytes,
                fetch_scale=f_scale, write_scale=w_scale,
                fetch_bytes=fetch_b, write_bytes=write_b, bytes_per_launch=fetch_b + write_b)


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("db", nargs="?")
    ap.add_argument("--kernel", default=None)
    ap.add_argument("--json", action="store_true")
    ap.add_argument("--traffic", nargs=4, metavar=("FETCH_DB", "WRITE_DB", "COPY_FETCH_DB", "COPY_WRITE_DB"))
    ap.add_argument("--copy-bytes", type=int, default=1 << 30)
    ap.add_argument("--workload", default="full")
    ap.add_argument("--out", default=None)
    a = ap.parse_args()
    if a.traffic:
        t = traffic(*a.traffic, kernel=a.kernel or "estimate_kernel", copy_bytes=a.copy_bytes,
                    workload=a.workload)
        txt = json.dumps(t, indent=1)
        if a.out:
            with open(a.out, "w") as fh:
                fh.write(txt + "\n")
        print(txt)
        return 0
    ds = dispatch_stats(a.db, a.kernel)
    cs = counter_stats(a.db, a.kernel)
    if a.json:
        print(json.dumps(dict(dispatches=ds, counters=cs,
                              kernel_source_sha=kernel_source_sha(a.kernel or "estimate_kernel"))))
        return 0
    if ds:
        print(f"{'calls':>6} {'total_us':>14} {'avg_us':>14} {'min_us':>14} {'max_us':>14}  kernel")
        for d in ds:
            print(f"{d['calls']:>6} {d['total_us']:>14.1f} {d['avg_us']:>14.1f} {d['min_us']:>14.1f} "
                  f"{d['max_us']:>14.1f}  {d['name'][:110]}")
    if cs:
        print(f"{'dispatches':>10} {'per_dispatch':>18}  counter  kernel")
        for c in cs:
            print(f"{c['dispatches']:>10} {c['per_dispatch']:>18.6g}  {c['counter']:<12} {c['name'][:100]}")
    return 0


if __name__ == "__main__":
    sys.exit(main())
