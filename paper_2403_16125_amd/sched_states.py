"""Seeded synthetic inputs for the scheduler that consumes the throughput
matrix: per-job throughput curves and cluster states.

This module only draws inputs (throughput values, allocations, queues and
priorities); it contains none of the scheduler's arithmetic, and both the HIP
path and the CPU oracle use it.  Random numbers: the SplitMix64 streams of
`workloads`.

Throughput curves follow the shape the paper reports for adaptive
parallelism (Sec. 2.3): zero below a job's smallest count that fits in
memory, then growing with the GPU count with diminishing returns, and faster
on faster GPU types.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .workloads import SplitMix64, _stream, _trace_counts


@dataclasses.dataclass
class SchedState:
    thr: np.ndarray           # f32 [J, T, NC] samples/s of job j on count c of type g (0: does not fit)
    counts: np.ndarray        # int32 [NC], strictly ascending
    capacity: np.ndarray      # int32 [T] GPUs of each type in the cluster
    alloc_type: np.ndarray    # int32 [J] type of a running job, -1 if not running
    alloc_count: np.ndarray   # int32 [J] count index of a running job
    queue: np.ndarray         # int32 [Q] pending job ids in queue order
    priority: np.ndarray      # int32 [Q] priority class of each queued job (smaller first)
    depth: int                # search depth D

    @property
    def n_jobs(self) -> int:
        return int(self.thr.shape[0])


def synthetic_thr(seed: int, n_jobs: int, n_types: int, counts) -> np.ndarray:
    """Throughput curves: thr = base * speed_g * n^alpha for n >= nmin, else 0."""
    counts = np.asarray(counts, np.int64)
    rng = SplitMix64(seed)
    speed = np.sort(rng.uniform_range(0.2, 1.0, n_types))[::-1]
    thr = np.zeros((n_jobs, n_types, len(counts)), np.float32)
    for j in range(n_jobs):
        r = _stream(seed, j)
        alpha = float(r.uniform_range(0.45, 0.95, 1)[0])
        base = float(np.exp(r.uniform_range(np.log(5.0), np.log(500.0), 1)[0]))
        nmin = int(r.choice(counts[: max(1, len(counts) // 2)], 1)[0])
        for g in range(n_types):
            fits = counts >= max(1, int(np.ceil(nmin / max(speed[g], 1e-9) ** 0.5)))
            curve = base * speed[g] * counts.astype(np.float64) ** alpha
            thr[j, g] = np.where(fits, curve, 0.0).astype(np.float32)
    return thr


def random_state(seed: int, thr: np.ndarray, counts, capacity, running_frac: float = 0.5,
                 queued_frac: float = 0.1, n_classes: int = 3, depth: int = 8,
                 max_count: int | None = None) -> SchedState:
    """A cluster state over the throughput matrix `thr`: a random share of jobs
    running on random feasible grids that fit the capacity (drawn in job
    order, with at most `max_count` GPUs if given), a random share queued with
    random priority classes."""
    J, T, NC = thr.shape
    counts = np.asarray(counts, np.int32)
    cap = np.asarray(capacity, np.int32)
    used = np.zeros(T, np.int64)
    rng = _stream(seed, 1 << 20)
    u = rng.uniform(3 * J)
    alloc_type = np.full(J, -1, np.int32)
    alloc_count = np.zeros(J, np.int32)
    queued = []
    for j in range(J):
        if u[3 * j] < running_frac:
            feas = [(g, c) for g in range(T) for c in range(NC)
                    if thr[j, g, c] > 0 and used[g] + counts[c] <= cap[g]
                    and (max_count is None or counts[c] <= max_count)]
            if feas:
                g, c = feas[int(u[3 * j + 1] * len(feas)) % len(feas)]
                alloc_type[j], alloc_count[j] = g, c
                used[g] += counts[c]
        elif u[3 * j] < running_frac + queued_frac:
            queued.append((int(u[3 * j + 2] * n_classes), j))
    queued.sort()
    return SchedState(thr=np.ascontiguousarray(thr, np.float32), counts=counts, capacity=cap,
                      alloc_type=alloc_type, alloc_count=alloc_count,
                      queue=np.asarray([j for _, j in queued], np.int32),
                      priority=np.asarray([p for p, _ in queued], np.int32), depth=int(depth))


def full_round(seed: int = 11) -> SchedState:
    """The scheduling step at the full-round size: the throughput matrix of
    16384 jobs x 8 GPU types x 131 GPU counts (powers of two and multiples of
    8 up to 1024), a 1280-GPU cluster (160 of each type, the size of the
    paper's simulated cluster), about half the jobs drawn as running on up to
    32 GPUs until the cluster is full, 2 % queued in 3 priority classes, and
    search depth 3 (the depth used in the paper's simulations)."""
    counts = np.asarray(_trace_counts(1024), np.int32)
    thr = synthetic_thr(seed, 16384, 8, counts)
    return random_state(seed, thr, counts, [160] * 8, running_frac=0.5, queued_frac=0.02,
                        n_classes=3, depth=3, max_count=32)


def deadlines(seed: int, thr: np.ndarray, slack=(0.8, 6.0), none_frac: float = 0.3):
    """Per-job batch, remaining iterations and seconds left to the deadline:
    batch from {64, 128, 256, 512}, iterations log-uniform on [1e3, 1e5], and
    the deadline the time to finish at the job's best throughput times a
    slack drawn uniformly from `slack` (below 1: no grid meets it); a share
    `none_frac` of jobs has no deadline (+inf)."""
    J = thr.shape[0]
    rng = _stream(seed, 1 << 21)
    u = rng.uniform(4 * J)
    batch = np.asarray([64, 128, 256, 512], np.int32)[(u[0::4] * 4).astype(np.int64) % 4]
    iters = np.exp(np.log(1e3) + u[1::4] * (np.log(1e5) - np.log(1e3))).astype(np.float32)
    best = thr.reshape(J, -1).max(axis=1).astype(np.float64)
    fac = slack[0] + u[2::4] * (slack[1] - slack[0])
    with np.errstate(divide="ignore"):
        ddl = np.where(best > 0, batch * iters.astype(np.float64) / np.where(best > 0, best, 1.0) * fac, 1.0)
    ddl = np.where(u[3::4] < none_frac, np.inf, ddl).astype(np.float32)
    return batch.astype(np.int32), iters, ddl
