"""Algorithmic work of one estimate: the numerator of the roofline fraction.

Counted is what the method must compute, independent of how a kernel
schedules it:

* a stage-partition problem is one (job, per-sample cost vector) pair.  The
  pure-compute vector (no tensor parallelism, no all-to-all) is the job's
  times divided by a scale, so it is one problem per job for every GPU type
  and count; every other vector is one per (job, type, tp, all-to-all flag,
  contention factor value);
* the problem's requested degrees S are the union over the cells sharing it
  and P its largest; the O(P L) bottleneck recursion fills P rows of L
  entries, 8 operations each (two subtracts, a compare, a min/max and an
  amortised pointer step);
* ops(problem) = 8 L (cost vector and prefix) + 8 L P (the recursion)
  + 4 L |S| (canonical cuts);
* ops(plan) = 12 pp + 40 (stage terms, memory check, reduction).

This is the convention the roofline fraction is quoted in (`ops`).  Two
smaller figures are kept beside it: `ops_truncated` counts only the entries
a recursion needs when row k stops at i = L - tau(k) + k (tau(k) the
smallest requested degree >= k), E = sum_{k=1}^{P} (L - tau(k) + 1); the
kernel's own tally counts the entries and plans it evaluated after bound
pruning.
"""
from __future__ import annotations

from functools import lru_cache

import numpy as np


def _divisors_upto(q: int, L: int):
    return [d for d in range(1, min(q, L) + 1) if q % d == 0]


@lru_cache(maxsize=None)
def _entries(L: int, targets: tuple) -> int:
    if not targets:
        return 0
    ts = sorted(targets)
    e, ti = 0, 0
    for k in range(1, ts[-1] + 1):
        while ts[ti] < k:
            ti += 1
        e += L - ts[ti] + 1
    return e


def count(w, kappa_round: int = 0) -> dict:
    """Exact algorithmic work of estimating every cell of workload `w`."""
    ms = [int(m) for m in w.m_values]
    kap = np.asarray(w.kappa[kappa_round], np.float32).reshape(w.n_types, w.n_counts)
    Ls = np.diff(w.layer_offset).astype(int)
    moe_job = np.zeros(w.n_jobs, bool)
    for j in range(w.n_jobs):
        moe_job[j] = bool((w.a2a[w.job_slice(j)] > 0).any())

    groups = {}
    for j in range(w.n_jobs):
        key = (int(Ls[j]), int(w.batch[j]), bool(moe_job[j]))
        groups[key] = groups.get(key, 0) + 1

    tot = dict(cells=w.n_cells, plans=0, plan_ops=0, problems=0, dp_entries=0, problem_ops=0,
               dp_entries_full=0, problem_ops_full=0)
    for (L, Bg, moe), mult in groups.items():
        pure_targets = set()
        shared = {}                  # (g, tp, flag, kappa) -> target set
        plans = plan_ops = 0
        for g in range(w.n_types):
            G = int(w.gpus_per_node[g])
            for ci, n in enumerate(int(c) for c in w.counts):
                kv = float(kap[g, ci])
                for tp in range(1, min(n, G) + 1):
                    if n % tp or G % tp:
                        continue
                    for pp in _divisors_upto(n // tp, L):
                        dp = n // (tp * pp)
                        nm = sum(1 for m in ms if Bg % (dp * m) == 0)
                        if not nm:
                            continue
                        plans += nm
                        plan_ops += nm * (12 * pp + 40)
                        a2a = moe and dp * tp > 1
                        if tp == 1 and not a2a:
                            pure_targets.add(pp)
                        else:
                            shared.setdefault((g, tp, a2a, kv), set()).add(pp)
        probs = [pure_targets] if pure_targets else []
        probs += list(shared.values())
        ent = sum(_entries(L, tuple(sorted(s))) for s in probs)
        ent_full = sum(L * max(s) for s in probs)
        base = sum(8 * L + 4 * L * len(s) for s in probs)
        pops = base + 8 * ent
        pops_full = base + 8 * ent_full
        tot["plans"] += mult * plans
        tot["plan_ops"] += mult * plan_ops
        tot["problems"] += mult * len(probs)
        tot["dp_entries"] += mult * ent
        tot["problem_ops"] += mult * pops
        tot["dp_entries_full"] += mult * ent_full
        tot["problem_ops_full"] += mult * pops_full
    tot["ops"] = tot["plan_ops"] + tot["problem_ops_full"]
    tot["ops_truncated"] = tot["plan_ops"] + tot["problem_ops"]
    return tot


# ------------------------------------------------------------ proxy planner

@lru_cache(maxsize=None)
def _pow2_splits(n: int, s: int, maxp: int) -> int:
    """Multisets of s powers of two (each <= maxp) summing to n."""
    if s == 0:
        return 1 if n == 0 else 0
    if n < s:
        return 0
    tot, p = 0, maxp
    while p >= 1:
        if p <= n - (s - 1):
            tot += _pow2_splits(n - p, s - 1, p)
        p //= 2
    return tot


@lru_cache(maxsize=None)
def _proxy_cell_ops(n: int, O: int, n_m: int) -> int:
    """Work of the proxy planner on one cell with O operators and n GPUs:
    every grouping of every grid normalised against every power-of-two
    multiset (3 fp64 ops -- subtract, multiply, add -- per stage and
    multiset), plus a memory test per stage and microbatch count (8 ops)."""
    from math import comb
    top = 1 << (n.bit_length() - 1)
    ops = 0
    for s in range(1, min(O, n) + 1):
        K = _pow2_splits(n, s, top)
        if K == 0:
            continue
        ops += comb(O - 1, s - 1) * (3 * s * K + 8 * s * n_m)
    return ops


def proxy_ops(w, n_ops: int = 16) -> int:
    """Algorithmic operations of one proxy-planner launch over every cell."""
    L = np.diff(np.asarray(w.layer_offset))
    per_job_ops = {}
    total = 0
    for Lj in L:
        O = int(min(int(Lj), n_ops))
        if O not in per_job_ops:
            per_job_ops[O] = sum(_proxy_cell_ops(int(n), O, len(w.m_values)) for n in w.counts)
        total += per_job_ops[O] * w.n_types
    return int(total)
