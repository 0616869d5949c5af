"""Benchmark: rebuild the job x grid throughput matrix of a full scheduling
round on one MI355X.

One step = one scheduling round: upload that round's per-grid contention
factors and estimate every (job, GPU type, GPU count) cell (16384 jobs x 8
types x 131 counts = 17.2 M cells, about 682 M plans).  Inputs are resident in
device memory before timing starts.  Prints one JSON line on stdout; progress
goes to stderr.

With --schedule it times instead the scheduling step that consumes such a
matrix (Algorithm 1 with the throughput objective, or with --objective
fairness the finish-time fairness objective) on a 1280-GPU cluster state over
the same 16384 x 8 x 131 shape, and prints that line.  With
--proxy it times the proxy-plan planner (Sec. 3.3) over every cell of the
trace-like workload and scores its plans against the exhaustive estimate.
With --partition memory the estimate prices each plan with the balanced
partition among the stage splits that fit memory instead of the balanced
partition followed by the memory check; with --partition exact-t on the split
of least iteration time among those that fit (trace-like workload: jobs of
at most 96 layers).  With --comm-tables communication
latency is interpolated in synthetic profiled (volume, latency) tables per
link instead of volume / bandwidth.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9   # CUs x SIMDs x lanes x clock: one unpacked VALU op per lane per clock
PUBLISHED_FP32 = 157.3e12                # MI355X fp32 vector, as published
COPY_BYTES = 1 << 30                    # calibration copy: 1 GiB read + 1 GiB written
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_estimate_full.json")


def stored_traffic(workload: str):
    """HBM bytes per estimate launch from the committed counter runs, if they
    were taken on the current kernel sources (else None)."""
    from paper_2403_16125_amd.rocprof_summary import kernel_source_sha
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha") != kernel_source_sha() or t.get("workload") != workload:
        return None
    return t.get("bytes_per_launch")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def host_info() -> dict:
    """The host the oracle is timed on: CPU model, the cores this process may
    use (capped at 16, the host share of one GPU), the oracle's compiler."""
    import platform
    import subprocess
    model = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    try:
        cc = subprocess.run(["gcc", "--version"], capture_output=True, text=True).stdout.splitlines()[0]
    except (OSError, IndexError):
        cc = "gcc"
    from oracle import oracle as oracle_c
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable,
            "threads": max(1, min(16, usable)), "compiler": cc, "flags": " ".join(oracle_c.CFLAGS)}


def _oracle_threads(fn, ids, threads: int) -> float:
    """Wall time of fn over ids split in `threads` contiguous chunks, one
    thread each (the oracle's C calls keep no global state and release the
    interpreter lock)."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    chunks = [c for c in np.array_split(ids, threads) if len(c)]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=len(chunks)) as ex:
        list(ex.map(fn, chunks))
    return time.perf_counter() - t0


def cpu_baseline(w, every: int, kappa_round: int = 0, rule: int = 0, tables=None, cell_every: int = 1) -> dict:
    """The oracle (C, fp64, one cell at a time) on a bounded sample of the
    same workload: jobs j = 0, every, 2*every, ... times every grid of one
    round, under partition rule `rule` or with communication latency from
    `tables`; timed on all usable host cores (jobs split over threads, each
    thread single-threaded code) and on one core."""
    import numpy as np
    from oracle import oracle as oracle_c
    oracle_c.load()
    info = host_info()
    per = w.n_types * w.n_counts
    jobs = list(range(0, w.n_jobs, every))
    ids = np.concatenate([np.arange(j * per, (j + 1) * per) for j in jobs]).astype(np.int64)[::cell_every]

    def run(sub):
        if tables is None:
            oracle_c.cells(w, sub, kappa_round=kappa_round, rule=rule)
        else:
            oracle_c.cells_tab(w, sub, tables, kappa_round=kappa_round)

    dt_all = _oracle_threads(run, ids, info["threads"])
    dt_one = _oracle_threads(run, ids, 1)
    return {"value": len(ids) / dt_all, "unit": "cells/s", "cores": info["threads"], "kind": "oracle",
            "sample": f"{len(jobs)} jobs (every {every}th) x {per} grids"
                      + (f", every {cell_every}th of those cells" if cell_every > 1 else "")
                      + f", contention round {kappa_round}: {len(ids)} cells, {dt_all:.1f} s on {info['threads']} "
                        f"threads, {dt_one:.1f} s on one",
            "single_core": {"value": len(ids) / dt_one, "unit": "cells/s", "cores": 1},
            "host": info}


def schedule_cpu_baseline(st, min_seconds: float = 10.0, objective: str = "throughput", work=None) -> dict:
    """The scheduler oracle (single-threaded Python) on the same state,
    repeated until about min_seconds of CPU work."""
    from oracle import scheduler_oracle as so
    kw = {} if work is None else dict(batch=work[0], iters=work[1])
    n, t0 = 0, time.perf_counter()
    while True:
        so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue,
                    st.priority, st.depth, objective=objective, **kw)
        n += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds and n >= 2:
            break
    return {"value": n / dt, "unit": "steps/s", "cores": 1, "kind": "oracle",
            "sample": f"the same state, {n} steps in {dt:.1f} s"}


def proxy_cpu_baseline(w, every: int, kappa_round: int = 0) -> dict:
    """The proxy-planner oracle (single-threaded C, fp64) on a bounded sample
    of the same workload: every `every`-th cell."""
    import numpy as np
    from oracle import proxy as proxy_c
    proxy_c.load()
    ids = np.arange(0, w.n_cells, every, dtype=np.int64)
    t0 = time.perf_counter()
    proxy_c.cells(w, ids, kappa_round=kappa_round)
    dt = time.perf_counter() - t0
    return {"value": len(ids) / dt, "unit": "cells/s", "cores": 1, "kind": "oracle",
            "sample": f"every {every}th cell of {args_workload_name(w)}: {len(ids)} cells in {dt:.1f} s"}


def args_workload_name(w) -> str:
    return f"{w.name} ({w.n_jobs} jobs x {w.n_types} types x {w.n_counts} counts)"


def bench_proxy(args) -> int:
    """One step = the proxy-plan planner (Sec. 3.3) over every cell of the
    workload (default: trace-like, 1024 jobs x 4 types x 35 counts); the
    exhaustive estimate of the same round scores its plans."""
    import numpy as np
    import torch

    from paper_2403_16125_amd import arena, workcount, workloads

    name = args.workload if args.workload != "full" or args.proxy_full else "trace"
    w = workloads.make(name)
    ops = workcount.proxy_ops(w, args.n_ops)
    log(f"proxy planner on {args_workload_name(w)}: {w.n_cells} cells, {ops:.4g} ops per launch")
    dev = torch.device("cuda", 0)
    est = arena.Estimator(w, device=0)
    stream = torch.cuda.current_stream(dev)
    for i in range(args.warmup):
        est.proxy_estimate(f_ref=workloads.F_REF, n_ops=args.n_ops)
        torch.cuda.synchronize(dev)
        log(f"warmup {i + 1}/{args.warmup} done")
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        est.proxy_estimate(f_ref=workloads.F_REF, n_ops=args.n_ops)
        ends[i].record(stream)
        torch.cuda.synchronize(dev)
        log(f"step {i + 1}/{args.steps}: {starts[i].elapsed_time(ends[i]):.1f} ms")
    wall = time.perf_counter() - t0
    launch_ms = [a.elapsed_time(b) for a, b in zip(starts, ends)]
    step_s = float(np.mean(launch_ms)) / 1e3
    pr = est.proxy_results()
    est.estimate()
    ex = est.results()
    est.close()
    both = np.isfinite(pr["t_iter"]) & np.isfinite(ex["t_iter"])
    ratio = ex["t_iter"][both].astype(np.float64) / pr["t_iter"][both].astype(np.float64)
    achieved = ops / step_s
    line = {
        "metric": "(job,grid) cells/sec (proxy planner)",
        "value": w.n_cells / step_s,
        "unit": "cells/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"{args_workload_name(w)}: {w.n_cells} cells, {args.n_ops} operators per job, "
                               "every pipeline degree and microbatch count"},
        "proxy_score": {
            "what": "exhaustive best T / proxy T per cell (1 = the proxy is as fast as the exhaustive optimum)",
            "mean": float(ratio.mean()), "median": float(np.median(ratio)),
            "frac_faster_than_exhaustive": float((ratio > 1).mean()),
            "cells": int(both.sum()),
            "proxy_only_feasible": int((np.isfinite(pr["t_iter"]) & ~np.isfinite(ex["t_iter"])).sum()),
        },
        "roofline": {
            "bound": "alu",
            "achieved": achieved / 1e12,
            "peak": PEAK_LANE_OPS / 1e12,
            "unit": "Top/s",
            "frac": achieved / PEAK_LANE_OPS,
            "traffic": None,
            "ops_per_launch": ops,
            "launch_ms": step_s * 1e3,
        },
    }
    if not args.no_cpu_baseline:
        log("timing the proxy oracle on a sample")
        line["cpu_baseline"] = proxy_cpu_baseline(w, args.proxy_cpu_every)
    log(f"timed {args.steps} launches in {wall:.2f} s wall")
    print(json.dumps(line), flush=True)
    return 0


def bench_schedule(args) -> int:
    """One step = one scheduling step (Algorithm 1, throughput or fairness
    objective) on the full-round state, from the same starting allocation
    every time."""
    import numpy as np
    import torch

    from paper_2403_16125_amd import arena, sched_states

    log("generating the full-round scheduler state")
    st = sched_states.full_round()
    J, T, NC = st.thr.shape
    log(f"{J} jobs x {T} types x {NC} counts, {int((st.alloc_type >= 0).sum())} running, "
        f"{len(st.queue)} queued, depth {st.depth}")
    dev = torch.device("cuda", 0)
    sch = arena.Scheduler(st.thr, st.counts, st.capacity, device=0, objective=args.objective)
    work = None
    if args.objective == "fairness":
        # each job's batch and remaining iterations (the deadline recipe's; no deadline)
        B, N, _ = sched_states.deadlines(11, st.thr, slack=(0.9, 4.0))
        work = (B, N)
        sch.set_deadlines(B, N, None)
    sch.load_state(st.alloc_type, st.alloc_count, st.queue, st.priority)
    at0, ac0 = sch.alloc_type.clone(), sch.alloc_count.clone()
    stream = torch.cuda.current_stream(dev)

    def reset():
        sch.alloc_type.copy_(at0)
        sch.alloc_count.copy_(ac0)

    for i in range(args.warmup):
        reset()
        sch.step(st.depth)
        torch.cuda.synchronize(dev)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for i in range(args.steps):
        reset()
        starts[i].record(stream)
        sch.step(st.depth)
        ends[i].record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    launch_ms = [a.elapsed_time(b) for a, b in zip(starts, ends)]
    res = sch.results()
    sch.close()
    if res["status"] != 0:
        log(f"schedule status {res['status']}")
        return 1
    step_s = float(np.mean(launch_ms)) / 1e3
    log(f"timed {args.steps} steps: {wall:.3f} s wall, kernel avg {step_s * 1e3:.3f} ms, "
        f"{res['decisions']} decisions, moves {res['moves']}")
    achieved = res["scanned"] / step_s
    line = {
        "metric": "scheduling steps/sec",
        "value": 1.0 / step_s,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": f"scheduling step over the full-round throughput matrix: {J} jobs x {T} GPU types "
                        f"x {NC} GPU counts, 1280-GPU cluster, {int((st.alloc_type >= 0).sum())} running, "
                        f"{len(st.queue)} queued in 3 classes, search depth {st.depth}",
            "objective": "throughput (Eq. 5)" if args.objective == "throughput" else
                         "finish-time fairness (Eq. 7)",
        },
        "decisions": res["decisions"],
        "ns_per_decision": step_s / max(1, res["decisions"]) * 1e9,
        "moves": {"scale_downs_kept": res["moves"][0], "launches": res["moves"][1],
                  "scale_ups": res["moves"][2]},
        "roofline": {
            "bound": "alu",
            "achieved": achieved / 1e12,
            "peak": PEAK_LANE_OPS / 1e12,
            "unit": "Top/s",
            "frac": achieved / PEAK_LANE_OPS,
            "traffic": None,
            "ops_per_launch": res["scanned"],
            "launch_ms": step_s * 1e3,
        },
    }
    if not args.no_cpu_baseline:
        log("timing the scheduler oracle on the same state")
        line["cpu_baseline"] = schedule_cpu_baseline(st, objective=args.objective, work=work)
    print(json.dumps(line), flush=True)
    return 0


VALU_OPS = (("fma", 1), ("add", 1), ("minmax", 2), ("select", 3))   # (class, operations per step)


def bench_valu_rate() -> int:
    """Issue rate of the estimate kernels' operation classes in fp64 and fp32
    (csrc/valu_rate.hip): 2048 blocks of 256 threads (eight waves per SIMD),
    eight independent chains per thread.  Prints one JSON line: per class and
    type, chain steps per second and their fp64 / fp32 ratio."""
    import ctypes
    from paper_2403_16125_amd import build
    lib = ctypes.CDLL(build.VALU_RATE_OUT)
    lib.valu_rate_run.restype = ctypes.c_int
    lib.valu_rate_run.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                  ctypes.POINTER(ctypes.c_double)]
    blocks, iters, reps = 2048, 32768, 5
    steps = blocks * 256 * 8 * iters                   # chain steps per launch
    out = {"what": "VALU issue rate: chain steps per second by operation class and type "
                   "(2048 x 256 threads, 8 independent chains each, no packed fp32)",
           "blocks": blocks, "iters": iters, "steps_per_launch": steps, "classes": {}}
    for op, (name, n_ops) in enumerate(VALU_OPS):
        row = {"ops_per_step": n_ops}
        for is_double, tname in ((1, "f64"), (0, "f32")):
            ms = (ctypes.c_double * reps)()
            rc = lib.valu_rate_run(op, is_double, blocks, iters, reps, ms)
            if rc != 0:
                print(f"valu_rate_run({name}, {tname}) failed: HIP error {rc}", file=sys.stderr, flush=True)
                return 1
            best = min(ms[i] for i in range(reps))
            row[tname] = {"ms": best, "steps_per_s": steps / (best * 1e-3)}
            log(f"{name} {tname}: {best:.3f} ms, {steps / (best * 1e-3):.4g} steps/s")
        row["f64_over_f32"] = row["f64"]["steps_per_s"] / row["f32"]["steps_per_s"]
        out["classes"][name] = row
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="full", choices=["tiny", "small", "trace", "moe", "full"])
    ap.add_argument("--cuts", action="store_true", help="also write the stage cuts of every cell")
    ap.add_argument("--cpu-every", type=int, default=None,
                    help="oracle sample: every k-th job (default 256; 2048 with --partition memory, "
                         "1024 with --comm-tables, 12 with --partition exact-t)")
    ap.add_argument("--partition", default="balanced", choices=["balanced", "memory", "exact-t"],
                    help="stage partition rule of the estimate (exact-t: the trace-like workload unless "
                         "--workload names another of at most 96 layers per job)")
    ap.add_argument("--comm-tables", action="store_true",
                    help="communication latency from synthetic profiled tables (interpolated by volume)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--schedule", action="store_true",
                    help="time the scheduling step that consumes the throughput matrix instead")
    ap.add_argument("--objective", default="throughput", choices=["throughput", "fairness"],
                    help="with --schedule, the scheduling objective")
    ap.add_argument("--proxy", action="store_true",
                    help="time the proxy-plan planner instead (trace-like workload unless --proxy-full)")
    ap.add_argument("--proxy-full", action="store_true", help="with --proxy, run it on the full round")
    ap.add_argument("--n-ops", type=int, default=16, help="operators per job for the proxy planner")
    ap.add_argument("--proxy-cpu-every", type=int, default=199, help="proxy oracle sample: every k-th cell")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain elementwise copy of known size (HBM counter calibration)")
    ap.add_argument("--valu-rate", action="store_true",
                    help="run only the fp64-vs-fp32 VALU issue-rate microbenchmark")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus} GPUs, WORLD_SIZE={world}): "
              "the estimator shards by job rows, but this benchmark measures a single GPU.",
              file=sys.stderr, flush=True)
        return 2

    if args.valu_rate:
        return bench_valu_rate()
    if args.schedule:
        return bench_schedule(args)
    if args.proxy:
        return bench_proxy(args)

    import numpy as np
    import torch

    from paper_2403_16125_amd import arena, workcount, workloads

    if args.copy_calibration:
        n = COPY_BYTES // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.mul(src, 1.0, out=dst)          # one elementwise kernel: reads and writes COPY_BYTES
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": COPY_BYTES}), flush=True)
        return 0

    if args.partition == "exact-t" and args.workload == "full":
        args.workload = "trace"             # the exact-T rule takes jobs of at most 96 layers
    log(f"generating workload {args.workload}")
    w = workloads.make(args.workload)
    log(f"{w.n_jobs} jobs, {w.n_types} types, {w.n_counts} counts, {w.n_cells} cells, "
        f"{w.n_rounds} rounds of contention factors")
    work = workcount.count(w, kappa_round=0)
    log(f"work per round (exhaustive plan space): {work['ops']:.4g} ops ({work['dp_entries_full']:.4g} recursion "
        f"entries), {work['plans']} plans, {work['problems']} partition problems; truncated rows "
        f"{work['ops_truncated']:.4g} ops")

    dev = torch.device("cuda", 0)
    rule = {"balanced": arena.PARTITION_BALANCED, "memory": arena.PARTITION_MEMORY,
            "exact-t": arena.PARTITION_EXACT_T}[args.partition]
    tables = workloads.comm_tables(w) if args.comm_tables else None
    if tables is not None and rule != arena.PARTITION_BALANCED:
        print("--comm-tables works with the balanced partition only", file=sys.stderr, flush=True)
        return 2
    est = arena.Estimator(w, device=0, with_cuts=args.cuts, rule=rule, comm_tables=tables)
    plain = rule == arena.PARTITION_BALANCED and tables is None
    size = est.space_size()
    assert size["plans"] == work["plans"]
    stream = torch.cuda.current_stream(dev)

    for i in range(args.warmup):
        est.set_round(i % w.n_rounds)
        est.estimate()
        torch.cuda.synchronize(dev)
        log(f"warmup {i + 1}/{args.warmup} done")

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for i in range(args.steps):
        est.set_round(i % w.n_rounds)
        starts[i].record(stream)
        est.estimate()
        ends[i].record(stream)
    torch.cuda.synchronize(dev)
    wall = time.perf_counter() - t0
    launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    avg_launch_s = float(np.mean(launch_ms)) / 1e3
    log(f"timed {args.steps} rounds: {wall:.3f} s wall, launch avg {avg_launch_s * 1e3:.2f} ms "
        f"(min {min(launch_ms):.2f}, max {max(launch_ms):.2f})")
    # the work each timed launch did (bound pruning depends on the round's
    # contention factors): the device tallies of the same rounds, re-run untimed
    ops_done, counts_done = [], []
    for i in range(args.steps):
        est.set_round(i % w.n_rounds)
        est.estimate()
        cnt = est.counters()
        ops_done.append(cnt["alg_ops"])
        counts_done.append(cnt)
    res = est.results(np.arange(0, w.n_cells, 9973))
    est.close()

    traffic = stored_traffic(args.workload) if plain else None
    cells_per_s = w.n_cells * args.steps / wall
    launch_s = float(np.sum(launch_ms)) / 1e3
    # numerator: the method's work per round over the exhaustive plan space (8 L + 8 L P
    # + 4 L |S| per distinct partition problem, 12 pp + 40 per plan); it does not
    # depend on the contention round.  Beside it: the same units with
    # truncated recursion rows, and the device's tally of the work it did.
    ops_round = float(work["ops"]) if plain else None
    achieved = ops_round * args.steps / launch_s if plain else float(np.sum(ops_done)) / launch_s
    tally_rate = float(np.sum(ops_done)) / launch_s
    priced = float(np.mean([c["plans"] for c in counts_done]))
    line = {
        "metric": "(job,grid) cells/sec",
        "value": cells_per_s,
        "unit": "cells/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: {w.n_jobs} jobs x {w.n_types} GPU types x {w.n_counts} GPU counts "
                        f"({w.n_cells} cells, {work['plans']} plans per round), per-grid contention "
                        "redrawn every round",
            "cuts": bool(args.cuts),
            "partition": args.partition,
            "comm": "interpolated tables" if tables is not None else "volume / bandwidth",
            "rounds_per_step": 1,
        },
        # every plan of the space is decided each round: priced, or skipped by
        # an exact bound
        "plans_decided_per_s": work["plans"] * args.steps / launch_s,
        "plans_priced_per_s": priced * args.steps / launch_s,
        "roofline": {
            "bound": "alu",
            "achieved": achieved / 1e12,
            "peak": PEAK_LANE_OPS / 1e12,
            "unit": "Top/s",
            "frac": achieved / PEAK_LANE_OPS,
            "traffic": traffic,
            "ops_per_launch": ops_round if plain else float(np.mean(ops_done)),
            "ops_convention": ("exhaustive: 8 L + 8 L P + 4 L |S| per distinct partition problem + 12 pp + 40 per plan"
                               if plain else "device tally of the work done"),
            "launch_ms": launch_s / args.steps * 1e3,
            "frac_truncated_rows": (float(work["ops_truncated"]) * args.steps / launch_s / PEAK_LANE_OPS
                                    if plain else None),
            "frac_device_tally": tally_rate / PEAK_LANE_OPS,
            "ops_device_tally": float(np.mean(ops_done)),
            # for transparency: against the published fp32 vector rate (FMA and packed pairs
            # counted twice each), and the measured HBM rate when the counters are current
            "frac_of_published_fp32": achieved / PUBLISHED_FP32,
            "hbm_GBps": (traffic / (launch_s / args.steps) / 1e9) if traffic else None,
        },
        "device_tallies": cnt,
        "feasible_fraction_sampled": float(np.mean(res["feasible"])),
    }
    if not args.no_cpu_baseline:
        log("timing the oracle on a sample")
        exact = rule == arena.PARTITION_EXACT_T
        every = args.cpu_every or (256 if plain else (12 if exact else (1024 if tables is not None else 2048)))
        line["cpu_baseline"] = cpu_baseline(w, every, rule=rule, tables=tables, cell_every=10 if exact else 1)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
