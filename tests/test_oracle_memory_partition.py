"""Pins of the oracle's memory-constrained stage partition (CPU only).

Under partition rule 1 a plan's stages are the balanced partition (the
slowest stage as fast as possible, Sec. 3.2) among the splits whose every
stage fits the GPU's memory (Sec. 3.3 picks parallelism within memory
limits); the memory of stage k of pp is 4 P_k/tp + min(m, pp-k) b A_k/tp.
The oracle finds it with a recursion over suffixes.  Fixed outside that
recursion here:
  * hand-worked partitions and cells, each derived in its comment;
  * brute force over every cut vector on small inputs (value and the
    lexicographically smallest optimal cuts);
  * special cases: unlimited memory gives the unconstrained partition, and a
    plan whose unconstrained partition fits keeps it;
  * invariants: more memory never raises the bottleneck, the cuts returned
    fit and attain it, and a cell's best time never rises against rule 0;
  * an enumeration of every plan and every cut vector of small cells.
"""
import itertools
import math

import numpy as np
import pytest

from paper_2403_16125_amd import workloads as wl

INF = math.inf


def _U(o, u):
    return o.prefix(np.asarray(u, np.float64))


# (u, p, a, pp, m, b, tp, mem) -> (W, cuts); derivations in the comments
HAND = [
    # weights only, m = 1: stage memory 4 P.  With mem 12 a stage holds P <= 3:
    # [0,1) has P 3 and [1,4) P 3; the balanced [0,2) would need 16.
    (dict(u=[1, 1, 1, 1], p=[3, 1, 1, 1], a=[0] * 4, pp=2, m=1, b=1.0, tp=1, mem=12.0), (3.0, [1])),
    # the same with tp = 2 and half the memory: everything divides by tp
    (dict(u=[1, 1, 1, 1], p=[3, 1, 1, 1], a=[0] * 4, pp=2, m=1, b=1.0, tp=2, mem=6.0), (3.0, [1])),
    # activations only, m = 2, pp = 3: stages 0 and 1 hold min(2, 3) = min(2, 2)
    # = 2 microbatches (A <= 1: one layer each), stage 2 holds 1 (A <= 2: two
    # layers).  The only split is [0,1) [1,2) [2,4): W = max(1, 1, 1 + 3) = 4,
    # against the unconstrained 3 with cuts [1, 3].
    (dict(u=[1, 1, 1, 3], p=[0] * 4, a=[1, 1, 1, 1], pp=3, m=2, b=1.0, tp=1, mem=2.0), (4.0, [1, 2])),
    # the same with b = 0.5 and half the memory
    (dict(u=[1, 1, 1, 3], p=[0] * 4, a=[1, 1, 1, 1], pp=3, m=2, b=0.5, tp=1, mem=1.0), (4.0, [1, 2])),
    # pp = 2 of the same: stage 0 holds 2 microbatches (one layer), stage 1 one
    # (two layers): three layers at most, no split of four fits
    (dict(u=[1, 1, 1, 3], p=[0] * 4, a=[1, 1, 1, 1], pp=2, m=2, b=1.0, tp=1, mem=2.0), (INF, None)),
    # more stages can be infeasible where fewer fit: a = [4, 1, 1, 1], m = 4,
    # mem 8.  pp = 1 holds one microbatch of A = 7; pp = 2: [0,1) holds 2 x 4,
    # [1,4) 1 x 3; pp = 3 and 4 put layer 0 alone first with 3 or 4 microbatches
    (dict(u=[2, 1, 1, 1], p=[0] * 4, a=[4, 1, 1, 1], pp=1, m=4, b=1.0, tp=1, mem=8.0), (5.0, [])),
    (dict(u=[2, 1, 1, 1], p=[0] * 4, a=[4, 1, 1, 1], pp=2, m=4, b=1.0, tp=1, mem=8.0), (3.0, [1])),
    (dict(u=[2, 1, 1, 1], p=[0] * 4, a=[4, 1, 1, 1], pp=3, m=4, b=1.0, tp=1, mem=8.0), (INF, None)),
    (dict(u=[2, 1, 1, 1], p=[0] * 4, a=[4, 1, 1, 1], pp=4, m=4, b=1.0, tp=1, mem=8.0), (INF, None)),
    # a stage exactly at the limit fits (<=): [0,2) holds 4 (1 + 1) = 8 weights
    (dict(u=[1, 1, 1, 1], p=[1, 1, 1, 1], a=[0] * 4, pp=2, m=1, b=1.0, tp=1, mem=8.0), (2.0, [2])),
    # zero-cost layers: lexicographically smallest among the fitting optima.
    # u = [0, 0, 3, 0]: every split has W = 3; stage 0 must stay P <= 1
    # (p = [1, 1, 0, 0], mem 4), so c_1 = 1 still fits and is smallest
    (dict(u=[0, 0, 3, 0], p=[1, 1, 0, 0], a=[0] * 4, pp=2, m=1, b=1.0, tp=1, mem=4.0), (3.0, [1])),
    # ... but with p = [0, 1, 1, 0]: c_1 = 1 leaves P 2 (8 > 4) on stage 1,
    # c_1 = 2 gives P 1 and 1, c_1 = 3 puts P 2 on stage 0: the cut moves to 2
    # at the same W
    (dict(u=[0, 0, 3, 0], p=[0, 1, 1, 0], a=[0] * 4, pp=2, m=1, b=1.0, tp=1, mem=4.0), (3.0, [2])),
]


@pytest.mark.parametrize("case,want", HAND, ids=[f"hand{i}" for i in range(len(HAND))])
def test_hand_worked(oracle, case, want):
    c = dict(case)
    U = _U(oracle, c.pop("u"))
    for brute in (False, True):
        w, cuts = oracle.bottleneck_mem(U, brute=brute, **c)
        assert w == want[0] and cuts == want[1], brute


def _random_instance(rng, L, zero_frac=0.0):
    u = rng.lognormal(0.0, 1.0, L)
    u[rng.random(L) < zero_frac] = 0.0
    u = np.round(u * 8) / 8              # repeated values: ties among cut vectors
    p = rng.lognormal(0.0, 1.0, L)
    a = rng.lognormal(0.0, 1.0, L)
    return u, p, a


def test_recursion_matches_bruteforce(oracle):
    rng = np.random.default_rng(7)
    n_fin = n_inf = 0
    for trial in range(500):
        L = int(rng.integers(1, 11))
        u, p, a = _random_instance(rng, L, zero_frac=0.2 if trial % 3 == 0 else 0.0)
        U = _U(oracle, u)
        pp = int(rng.integers(1, L + 1))
        m = int(rng.choice([1, 2, 3, 8]))
        tp = int(rng.choice([1, 2, 4]))
        b = float(rng.choice([0.25, 1.0, 3.0]))
        # the memory of the whole model on one stage, scaled: binds often
        whole = (4.0 * p.sum() + min(m, pp) * b * a.sum()) / tp
        mem = float(whole * rng.uniform(0.15, 1.1) / max(1, pp // 2))
        wd, cd = oracle.bottleneck_mem(U, p, a, pp, m, b, tp, mem)
        wb, cb = oracle.bottleneck_mem(U, p, a, pp, m, b, tp, mem, brute=True)
        assert wd == wb and cd == cb, (trial, L, pp, m, tp, b, mem)
        n_fin += math.isfinite(wd)
        n_inf += not math.isfinite(wd)
    assert n_fin > 150 and n_inf > 50    # both outcomes well represented


def test_unlimited_memory_is_the_unconstrained_partition(oracle):
    rng = np.random.default_rng(3)
    for L in (1, 2, 5, 17, 64, 128):
        u, p, a = _random_instance(rng, L, zero_frac=0.1)
        U = _U(oracle, u)
        for pp in sorted(q for q in {1, 2, 3, L // 2 or 1, L} if q <= L):
            w, cuts = oracle.bottleneck_mem(U, p, a, pp, 4, 2.0, 2, INF)
            w0 = oracle.bottleneck_dp(U, pp)
            assert w == w0
            assert cuts == oracle.canonical_cuts(U, pp, w0)


def _stage_mem(p, a, cuts, pp, m, b, tp):
    # memory of each stage, summed in the model's order (independent of the oracle's code)
    bounds = [0] + list(cuts) + [len(p)]
    out = []
    for k in range(pp):
        P = 0.0
        A = 0.0
        for l in range(bounds[k], bounds[k + 1]):
            P += float(p[l])
            A += float(a[l])
        out.append(4.0 * P / tp + min(m, pp - k) * b * A / tp)
    return out


def test_fitting_unconstrained_partition_is_kept_and_results_fit(oracle):
    rng = np.random.default_rng(11)
    kept = moved = 0
    for trial in range(300):
        L = int(rng.integers(2, 40))
        u, p, a = _random_instance(rng, L)
        U = _U(oracle, u)
        pp = int(rng.integers(1, L + 1))
        m, tp, b = int(rng.choice([1, 2, 4, 8])), int(rng.choice([1, 2])), float(rng.choice([0.5, 1.0, 2.0]))
        whole = (4.0 * p.sum() + min(m, pp) * b * a.sum()) / tp
        mem = float(whole * rng.uniform(0.2, 1.2) / max(1, pp // 2))
        w0 = oracle.bottleneck_dp(U, pp)
        c0 = oracle.canonical_cuts(U, pp, w0)
        w, cuts = oracle.bottleneck_mem(U, p, a, pp, m, b, tp, mem)
        assert w >= w0
        if max(_stage_mem(p, a, c0, pp, m, b, tp)) <= mem:
            assert w == w0 and cuts == c0
            kept += 1
        elif math.isfinite(w):
            moved += 1
        if math.isfinite(w):
            # the returned cuts fit and attain W
            assert max(_stage_mem(p, a, cuts, pp, m, b, tp)) <= mem
            bounds = [0] + cuts + [L]
            assert max(U[bounds[k + 1]] - U[bounds[k]] for k in range(pp)) == w
            assert all(bounds[k] < bounds[k + 1] for k in range(pp))
    assert kept > 30 and moved > 30


def test_more_memory_never_raises_the_bottleneck(oracle):
    rng = np.random.default_rng(5)
    for trial in range(120):
        L = int(rng.integers(2, 48))
        u, p, a = _random_instance(rng, L)
        U = _U(oracle, u)
        pp = int(rng.integers(1, L + 1))
        m = int(rng.choice([1, 2, 4]))
        whole = 4.0 * p.sum() + min(m, pp) * a.sum()
        prev = INF
        for f in np.linspace(0.05, 1.5, 12):
            w, _ = oracle.bottleneck_mem(U, p, a, pp, m, 1.0, 1, float(whole * f))
            assert w <= prev
            prev = w


# ---------------------------------------------------------------- cell level

def _cell(job, ty, n, m_values):
    return wl.from_lists([job], [ty], [n], m_values, kappa=1.0)


def test_hand_cell_weights():
    """Four layers of equal time (t = 1 for the whole batch of 1), weights
    3, 1, 1, 1 GB, no activations or comm; one GPU per node, 2 GPUs, m = 1.
    The only plan is (dp, tp, pp, m) = (1, 1, 2, 1) with b = 1.
    Rule 0: balanced cuts [2] put 4 GB of weights (16 GB) on stage 0 > 12 GB:
    the cell is infeasible.  Rule 1: cuts [1]: stages of 3 GB each (12 GB,
    fits), stage times 1 and 3: T = (1 + 3) + 0 x 3 = 4, throughput 1/4."""
    from oracle import oracle as o
    job = dict(t=[1, 1, 1, 1], p=[3e9, 1e9, 1e9, 1e9], a=[0] * 4, x=[0] * 4, a2a=[0] * 4, batch=1)
    ty = dict(speed=1.0, mem=12e9, bw_intra=1e9, bw_inter=1e9, gpus_per_node=1)
    w = _cell(job, ty, 2, [1])
    r0 = o.cells(w, [0], rule=0)
    assert r0["T"][0] == INF and r0["thr"][0] == 0.0 and r0["pp"][0] == 0
    r1 = o.cells(w, [0], rule=1)
    assert (r1["dp"][0], r1["tp"][0], r1["pp"][0], r1["m"][0]) == (1, 1, 2, 1)
    assert r1["T"][0] == 4.0 and r1["thr"][0] == 0.25
    assert list(r1["cuts"][0][:2]) == [1, -1]


def test_hand_cell_activations():
    """Layer times u = [1, 1, 1, 3] per sample (t = 2, 2, 2, 6 for the batch of
    2), activations 1 GB per sample each, no weights or comm, mem 2 GB; one GPU
    per node, 3 GPUs, m = 2.  Plans: pp = 1 needs dp = 3 (3 x 2 does not divide
    2); pp = 3, dp = 1, m = 2, b = 1.  Stages 0, 1, 2 hold 2, 2, 1
    microbatches.  Rule 0: balanced cuts [1, 3] give stage 1 two layers (4 GB):
    infeasible.  Rule 1: cuts [1, 2], stage times 1, 1, 4:
    T = (1 + 1 + 4) + (2 - 1) x 4 = 10, throughput 2/10."""
    from oracle import oracle as o
    job = dict(t=[2, 2, 2, 6], p=[0] * 4, a=[1e9] * 4, x=[0] * 4, a2a=[0] * 4, batch=2)
    ty = dict(speed=1.0, mem=2e9, bw_intra=1e9, bw_inter=1e9, gpus_per_node=1)
    w = _cell(job, ty, 3, [2])
    assert o.cells(w, [0], rule=0)["T"][0] == INF
    r1 = o.cells(w, [0], rule=1)
    assert (r1["dp"][0], r1["tp"][0], r1["pp"][0], r1["m"][0]) == (1, 1, 3, 2)
    assert r1["T"][0] == 10.0 and r1["thr"][0] == pytest.approx(0.2, rel=1e-15)
    assert list(r1["cuts"][0][:3]) == [1, 2, -1]


def _enumerate_cell(o, w, ci, tie_eps):
    """Every plan of the cell and every cut vector, priced with explicit cuts;
    per plan the fitting vectors with the least slowest stage, the
    lexicographically first; then the cell's choice (smallest (pp, tp, m)
    within the tie window of the least T)."""
    n = int(w.counts[ci])
    L = int(w.layer_offset[1] - w.layer_offset[0])
    gpn = int(w.gpus_per_node[0])
    bg = int(w.batch[0])
    kap = float(w.kappa[0][ci])
    cands = []
    for tp in range(1, n + 1):
        if n % tp or tp > gpn or gpn % tp:
            continue
        for pp in range(1, n // tp + 1):
            if (n // tp) % pp or pp > L:
                continue
            dp = n // (tp * pp)
            for m in w.m_values:
                m = int(m)
                if bg % (dp * m):
                    continue
                best = None
                for cuts in itertools.combinations(range(1, L), pp - 1):
                    e = o.eval_plan(w, 0, 0, n, kap, dp, tp, pp, m, cuts=list(cuts))
                    if not e["feasible"]:
                        continue
                    if best is None or e["s_max"] < best[0]:
                        best = (e["s_max"], e["T"], list(cuts))
                if best is not None:
                    cands.append((best[1], pp, tp, m, dp, best[2]))
    if not cands:
        return None
    tmin = min(c[0] for c in cands)
    win = min((c for c in cands if c[0] <= tmin * (1 + tie_eps)), key=lambda c: (c[1], c[2], c[3]))
    return win


def test_small_cells_against_enumeration(oracle):
    rng = np.random.default_rng(21)
    checked = differs = 0
    for trial in range(40):
        L = int(rng.integers(3, 9))
        job = dict(t=list(rng.lognormal(0, 0.7, L) * 8), p=list(rng.lognormal(20, 1.0, L)),
                   a=list(rng.lognormal(18, 1.0, L)), x=list(rng.lognormal(15, 0.5, L)),
                   a2a=[0.0] * L, batch=int(rng.choice([4, 8, 16])))
        tot = 4 * sum(job["p"]) + job["batch"] * sum(job["a"])
        ty = dict(speed=1.0, mem=float(tot * rng.uniform(0.08, 0.5)), bw_intra=2e11, bw_inter=2.5e10,
                  gpus_per_node=int(rng.choice([1, 2, 4])))
        counts = [1, 2, 3, 4, 6, 8]
        w = wl.from_lists([job], [ty], counts, [1, 2, 4, 8], kappa=1.0)
        ids = list(range(len(counts)))
        r1 = oracle.cells(w, ids, rule=1)
        r0 = oracle.cells(w, ids, rule=0)
        for ci in ids:
            want = _enumerate_cell(oracle, w, ci, float(w.tie_eps))
            checked += 1
            if want is None:
                assert r1["T"][ci] == INF and r1["pp"][ci] == 0
                continue
            T, pp, tp, m, dp, cuts = want
            assert (r1["dp"][ci], r1["tp"][ci], r1["pp"][ci], r1["m"][ci]) == (dp, tp, pp, m)
            assert r1["T"][ci] == T
            assert list(r1["cuts"][ci][:pp - 1]) == cuts
            # rule 1 never does worse than rule 0
            assert r1["T"][ci] <= r0["T"][ci]
            differs += r1["T"][ci] != r0["T"][ci]
    assert checked == 240 and differs > 10


def test_plans_of_workloads_keep_fitting_partitions(oracle):
    """On the synthetic workloads: a plan whose balanced partition fits keeps
    it (same T, same cuts); one that did not fit but now does is priced with
    cuts that fit; cells never get slower."""
    for name, step in (("trace", 3001), ("moe", 997)):
        w = wl.make(name)
        C = w.n_jobs * w.n_types * w.n_counts
        ids = np.arange(0, C, step)
        r0, r1 = oracle.cells(w, ids, rule=0), oracle.cells(w, ids, rule=1)
        f0 = np.isfinite(r0["T"])
        assert np.all(np.isfinite(r1["T"][f0]))
        assert np.all(r1["T"][f0] <= r0["T"][f0])
        for s in range(0, len(ids), 7):
            c = int(ids[s])
            ci = c % w.n_counts
            g = (c // w.n_counts) % w.n_types
            j = c // (w.n_counts * w.n_types)
            if not np.isfinite(r1["T"][s]):
                continue
            n = int(w.counts[ci])
            kap = float(w.kappa[0][g * w.n_counts + ci])
            plan = (int(r1["dp"][s]), int(r1["tp"][s]), int(r1["pp"][s]), int(r1["m"][s]))
            e0 = oracle.eval_plan(w, j, g, n, kap, *plan, rule=0)
            e1 = oracle.eval_plan(w, j, g, n, kap, *plan, rule=1)
            assert e1["feasible"] and e1["T"] == r1["T"][s]
            if e0["feasible"]:
                assert e0["T"] == e1["T"] and e0["cuts"] == e1["cuts"]
            ex = oracle.eval_plan(w, j, g, n, kap, *plan, cuts=e1["cuts"])
            assert ex["feasible"] and ex["T"] == e1["T"]
