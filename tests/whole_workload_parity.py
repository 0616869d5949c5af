"""Every cell of a whole workload -- by default the full scheduling round
(16384 jobs x 8 GPU types x 131 GPU counts = 17,170,432 cells) -- estimated
on the GPU and compared with the CPU oracle, cell by cell.

A script rather than a pytest case: the oracle needs about 4,700 core-seconds
for the full round, so it runs on every host core (threads; the oracles' C
calls release the interpreter lock and keep no global state) and takes
minutes.

    python tests/whole_workload_parity.py [--workload full|trace|moe] [--round R]
        [--partition balanced|memory|exact-t | --comm-tables | --proxy] [--threads N]

--partition memory, --partition exact-t (jobs of at most 96 layers: the
trace-like workload) and --comm-tables compare the estimator's variants with
the oracle's; --proxy compares the proxy-plan planner with its oracle (plan
identical -- stage count, microbatches, stage bounds, GPUs and tensor degree
per stage -- and T within 1e-6 relative).

The agreement rule is the one of the sampled parity tests (tests/compare.py):
same plan (dp, tp, pp, m) and stage cuts, iteration time and throughput within
1e-5 relative; a cell whose decision differs passes only as a near-tie (the
GPU's plan, priced by the oracle with the GPU's cuts, within 1e-5 of the
oracle's best or on the memory limit).  The bulk test is vectorised; only the
cells it does not settle go through the per-cell comparison.  Prints one
summary line and exits non-zero on any mismatch or on more than 1e-3 of the
cells as near-ties.
"""
from __future__ import annotations

import argparse
import os
import sys
import threading
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

REL = 1e-5


def say(*a):
    print("[full-parity]", *a, flush=True)


def settle(gpu, ref, lo, hi):
    """Vectorised exact test of cells [lo, hi): True where the GPU cell equals
    the oracle's (or both are the infeasible sentinel)."""
    g_feas = gpu["feasible"][lo:hi].astype(bool)
    o_feas = np.isfinite(ref["T"])
    t = gpu["t_iter"][lo:hi].astype(np.float64)
    thr = gpu["thr"][lo:hi].astype(np.float64)
    both_inf = ~g_feas & ~o_feas & np.isinf(t) & (thr == 0) & (gpu["dp"][lo:hi] == 0)
    if gpu.get("cuts") is not None:
        gc = gpu["cuts"][lo:hi].astype(np.int32)
        oc = ref["cuts"]
        both_inf &= (gc == 0xFF).all(axis=1)
        pp = gpu["pp"][lo:hi].astype(np.int32)
        col = np.arange(gc.shape[1], dtype=np.int32)[None, :]
        inside = col < (pp - 1)[:, None]
        cuts_ok = np.where(inside, gc == oc[:, :gc.shape[1]], gc == 0xFF).all(axis=1)
    else:                                # the timed launch writes no cut rows
        cuts_ok = np.ones(hi - lo, bool)
    with np.errstate(invalid="ignore", divide="ignore"):
        relT = np.abs(t - ref["T"]) / ref["T"]
        relthr = np.abs(thr - ref["thr"]) / ref["thr"]
    same = (g_feas & o_feas
            & (gpu["dp"][lo:hi] == ref["dp"]) & (gpu["tp"][lo:hi] == ref["tp"])
            & (gpu["pp"][lo:hi] == ref["pp"]) & (gpu["m"][lo:hi] == ref["m"])
            & cuts_ok & (relT <= REL) & (relthr <= REL))
    return both_inf | same, np.where(same, relT, 0.0)


def proxy_mismatches(got, want, lo, hi):
    """Cells [lo, hi) of the proxy planner whose plan or T differ from the oracle's."""
    bad = []
    for q in range(hi - lo):
        g = lo + q
        T = float(want["T"][q])
        if not np.isfinite(T):
            if got["feasible"][g] or np.isfinite(got["t_iter"][g]) or got["thr"][g] != 0 or got["words"][g].any():
                bad.append((g, "infeasible cell with outputs"))
            continue
        s = int(want["s"][q])
        mask = 0
        for b in want["bounds"][q][1:s]:
            mask |= 1 << (int(b) - 1)
        same = (got["feasible"][g] and int(got["s"][g]) == s and int(got["B"][g]) == int(want["B"][q])
                and int(got["starts"][g]) == mask
                and list(got["Dn"][g][:s]) == list(want["Dn"][q][:s])
                and list(got["tp"][g][:s]) == list(want["tp"][q][:s]))
        if not same:
            bad.append((g, "plan differs"))
        elif abs(float(got["t_iter"][g]) - T) > 1e-6 * T or \
                abs(float(got["thr"][g]) - float(want["thr"][q])) > 1e-6 * float(want["thr"][q]):
            bad.append((g, "T differs"))
    return bad


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="full", choices=["full", "trace", "moe"])
    ap.add_argument("--round", type=int, default=0, help="contention round (0..9)")
    ap.add_argument("--partition", default="balanced", choices=["balanced", "memory", "exact-t"])
    ap.add_argument("--comm-tables", action="store_true")
    ap.add_argument("--proxy", action="store_true")
    ap.add_argument("--no-cuts", action="store_true",
                    help="estimate without cut rows, as bench.py times it (plans, T, throughput compared)")
    ap.add_argument("--job-every", type=int, default=1,
                    help="compare the cells of every k-th job only (all grids of each); the GPU still "
                         "estimates the whole workload")
    ap.add_argument("--threads", type=int, default=min(16, os.cpu_count() or 1))
    ap.add_argument("--chunk-jobs", type=int, default=None,
                    help="jobs per oracle call (default 32; 4 with --partition memory, 2 with --partition "
                         "exact-t and --proxy, whose oracles are slower)")
    args = ap.parse_args()
    if sum([args.partition != "balanced", args.comm_tables, args.proxy]) > 1:
        ap.error("choose one of --partition memory|exact-t, --comm-tables, --proxy")

    from oracle import oracle
    from oracle import proxy as px
    from paper_2403_16125_amd import arena
    from paper_2403_16125_amd import workloads as wl
    from compare import compare, select

    oracle.load()
    w = wl.make(args.workload)
    rule = {"balanced": 0, "memory": 1, "exact-t": 2}[args.partition]
    tables = wl.comm_tables(w) if args.comm_tables else None
    mode = ("proxy planner" if args.proxy else "memory rule" if rule == 1 else "exact-T rule" if rule == 2 else
            "comm tables" if tables is not None else "balanced")
    say(f"{args.workload} round {args.round} ({mode}): {w.n_cells} cells; estimating on the GPU")
    est = arena.Estimator(w, with_cuts=not (args.proxy or args.no_cuts),
                          rule=(arena.PARTITION_BALANCED, arena.PARTITION_MEMORY, arena.PARTITION_EXACT_T)[rule],
                          comm_tables=tables)
    try:
        if args.round:
            est.set_round(args.round)
        if args.proxy:
            est.proxy_estimate(f_ref=wl.F_REF, n_ops=16)
            gpu = est.proxy_results()
        else:
            est.estimate()
            gpu = est.results()
    finally:
        est.close()
    per_job = w.n_types * w.n_counts
    if args.chunk_jobs is None:          # about 10-30 s of oracle work per chunk
        args.chunk_jobs = 2 if args.proxy or rule == 2 else 4 if rule else 32
    jobs = np.arange(0, w.n_jobs, args.job_every, dtype=np.int64)
    chunks = [jobs[i:i + args.chunk_jobs] for i in range(0, len(jobs), args.chunk_jobs)]
    n_want = len(jobs) * per_job
    say(f"GPU done; oracle on {args.threads} threads, {len(chunks)} chunks of {args.chunk_jobs} jobs")

    lock = threading.Lock()
    tot = dict(n=0, exact=0, near_tie=0, infeasible=0, max_rel_T=0.0, mismatch=[])
    done = [0]
    t0 = time.perf_counter()

    def work(ch):
        ids = (ch[:, None] * per_job + np.arange(per_job, dtype=np.int64)[None, :]).ravel()
        lo, hi = 0, len(ids)
        sub_gpu = {k: (v[ids] if v is not None else None) for k, v in gpu.items()}
        if args.proxy:
            want = px.cells(w, ids, kappa_round=args.round, f_ref=wl.F_REF, n_ops=16)
            bad = proxy_mismatches(sub_gpu, want, lo, hi)
            fin = np.isfinite(want["T"])
            relT = np.zeros(hi - lo)
            relT[fin] = np.abs(sub_gpu["t_iter"][fin].astype(np.float64) - want["T"][fin]) / want["T"][fin]
            ok = np.ones(hi - lo, bool)
            for g, _ in bad:
                ok[g - lo] = False
            rep = dict(exact=0, near_tie=0, max_rel_T=0.0, mismatch=[(int(ids[g]), why) for g, why in bad])
            ref = want
        else:
            ref = (oracle.cells(w, ids, kappa_round=args.round, rule=rule) if tables is None else
                   oracle.cells_tab(w, ids, tables, kappa_round=args.round))
            ok, relT = settle(sub_gpu, ref, lo, hi)
            rest = np.nonzero(~ok)[0]
            rep = None
            if len(rest):
                sub = {k: v[rest] for k, v in ref.items()}
                rep = compare(w, select(sub_gpu, rest), ids[rest], oracle, kappa_round=args.round, ref=sub,
                              rule=rule, tables=tables)
        n_inf = int((~np.isfinite(ref["T"])).sum())
        with lock:
            tot["n"] += hi - lo
            tot["exact"] += int(ok.sum()) + (rep["exact"] if rep else 0)
            tot["near_tie"] += rep["near_tie"] if rep else 0
            tot["infeasible"] += n_inf
            tot["max_rel_T"] = max(tot["max_rel_T"], float(relT.max(initial=0.0)),
                                   rep["max_rel_T"] if rep else 0.0)
            if rep:
                tot["mismatch"] += rep["mismatch"]
            done[0] += 1
            if done[0] % max(1, len(chunks) // 32) == 0 or done[0] == len(chunks):
                el = time.perf_counter() - t0
                say(f"{done[0]}/{len(chunks)} chunks, {tot['n']} cells, {el:.0f} s, "
                    f"near_tie={tot['near_tie']} mismatch={len(tot['mismatch'])}")

    with ThreadPoolExecutor(max_workers=args.threads) as ex:
        for f in [ex.submit(work, ch) for ch in chunks]:
            f.result()
    el = time.perf_counter() - t0
    sample = "" if args.job_every == 1 else f", one job in {args.job_every}"
    say(f"{args.workload} round {args.round} ({mode}{sample}): n={tot['n']} exact={tot['exact']} near_tie={tot['near_tie']} "
        f"mismatch={len(tot['mismatch'])} infeasible={tot['infeasible']} max_rel_T={tot['max_rel_T']:.3g} "
        f"oracle {el:.0f} s on {args.threads} threads")
    if tot["mismatch"]:
        say("first mismatches:", tot["mismatch"][:8])
    bad = bool(tot["mismatch"]) or tot["near_tie"] > 1e-3 * tot["n"] or tot["n"] != n_want
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(main())
