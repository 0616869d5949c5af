"""Parity of the exact-T partition rule (ARENA_PARTITION_EXACT_T) with the
oracle, through the C ABI on the GPU: every cell of the tiny and small
workloads and of the edge shapes, sampled trace-like cells (with two whole
jobs), the hand-derived plan, bound pruning on and off, and the jobs the rule
refuses.  Every case prints what it runs first."""
import sys

import numpy as np
import pytest

from paper_2403_16125_amd import arena
from paper_2403_16125_amd import workloads as wl

from compare import compare, oracle_cells_parallel

pytestmark = pytest.mark.gpu
RULE = arena.PARTITION_EXACT_T


def _say(*a):
    print("[exact-t]", *a, flush=True)
    sys.stdout.flush()


def _run(w, ids=None, prune=True, with_cuts=True):
    est = arena.Estimator(w, with_cuts=with_cuts, rule=RULE, prune=prune)
    try:
        est.estimate()
        res = est.results(ids)
        cnt = est.counters()
        size = est.space_size()
    finally:
        est.close()
    return res, cnt, size


def _check(rep, name):
    _say(f"{name}: n={rep['n']} exact={rep['exact']} near_tie={rep['near_tie']} "
         f"mismatch={len(rep['mismatch'])} infeasible={rep['infeasible']} max_rel_T={rep['max_rel_T']:.3g}")
    assert not rep["mismatch"], rep["mismatch"][:5]
    assert rep["near_tie"] <= max(2, 1e-3 * rep["n"])


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_every_cell(oracle, name):
    w = wl.make(name)
    _say(f"{name}: {w.n_cells} cells, all compared")
    res, cnt, size = _run(w)
    ids = np.arange(w.n_cells)
    ref = oracle_cells_parallel(oracle, w, ids, rule=RULE)
    _check(compare(w, res, ids, oracle, rule=RULE, ref=ref), name)
    assert cnt["cells"] == w.n_cells
    assert cnt["plans"] + cnt["plans_skipped"] == size["plans"]


def test_trace_sampled(oracle):
    w = wl.make("trace")
    rng = np.random.default_rng(31)
    ids = set(rng.choice(w.n_cells, 200, replace=False).tolist())
    per = w.n_types * w.n_counts
    for j in rng.choice(w.n_jobs, 2, replace=False):
        ids.update(range(int(j) * per, int(j) * per + per))
    ids = np.asarray(sorted(ids), np.int64)
    _say(f"trace: {w.n_cells} cells on the GPU, {len(ids)} compared")
    res, cnt, size = _run(w, ids=ids)
    ref = oracle_cells_parallel(oracle, w, ids, rule=RULE)
    _check(compare(w, res, ids, oracle, rule=RULE, ref=ref), "trace")
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]


def _edge():
    rng = np.random.default_rng(12)
    jobs = [dict(t=[2e-3], p=[1e8], a=[1e6], x=[1e5], a2a=[0.0], batch=8),
            dict(t=[0.0, 1e-3, 0.0, 0.0, 2e-3], p=[1e8, 0.0, 3e8, 1e8, 2e8], a=[1e6] * 5,
                 x=[1e5, 4e5, 1e5, 2e5, 1e5], a2a=[0.0] * 5, batch=16),
            dict(t=list(rng.uniform(1e-3, 2e-3, 40)), p=list(rng.uniform(1e7, 4e8, 40)), a=[2e6] * 40,
                 x=list(rng.uniform(1e4, 4e5, 40)), a2a=[0.0] * 40, batch=64),
            dict(t=list(rng.lognormal(-6, 0.8, 96)), p=list(rng.uniform(1e8, 3e8, 96)), a=[4e6] * 96,
                 x=[2.5e5] * 96, a2a=[0.0 if i % 2 == 0 else 4e5 for i in range(96)], batch=128),
            dict(t=[1e-3] * 24, p=[1e10] * 24, a=[1e9] * 24, x=[1e7] * 24, a2a=[0.0] * 24, batch=4)]
    types = [dict(speed=1.0, mem=80e9, bw_intra=300e9, bw_inter=25e9, gpus_per_node=8),
             dict(speed=0.5, mem=16e9, bw_intra=np.inf, bw_inter=np.inf, gpus_per_node=1),
             dict(speed=0.7, mem=12e9, bw_intra=64e9, bw_inter=12.5e9, gpus_per_node=16)]
    counts = [1, 2, 3, 8, 24, 96]
    return wl.from_lists(jobs, types, counts, [1, 2, 4, 8, 16, 32, 64],
                         kappa=rng.uniform(1.0, 2.0, len(types) * len(counts)))


def test_edge_shapes(oracle):
    w = _edge()
    _say(f"edge: {w.n_cells} cells, all compared")
    res, cnt, size = _run(w)
    ids = np.arange(w.n_cells)
    rep = compare(w, res, ids, oracle, rule=RULE, ref=oracle_cells_parallel(oracle, w, ids, rule=RULE))
    _check(rep, "edge")
    assert rep["infeasible"] > 0 and res["pp"].max() >= 24


def test_hand_plan():
    # four layers of equal cost, parameters in the last two, dp = 2, m = 2 on one
    # node of 4 GPUs with 4 B/s links: the balanced split (after layer 2) costs
    # 10, the exact-T split (after layer 3) costs 9 (worked out in the oracle pins)
    job = dict(t=[4.0] * 4, p=[0.0, 0.0, 8.0, 8.0], a=[0.0] * 4, x=[0.0] * 4, a2a=[0.0] * 4, batch=4)
    ty = dict(speed=1.0, mem=1e12, bw_intra=4.0, bw_inter=4.0, gpus_per_node=1)
    # gpus_per_node 1: tp = 1 only, so the plans of 4 GPUs are dp x pp = 4
    w = wl.from_lists([job], [ty], [4], [2], kappa=1.0)
    _say("hand plan")
    res, _, _ = _run(w)
    est = arena.Estimator(w, with_cuts=True, rule=arena.PARTITION_BALANCED)
    try:
        est.estimate()
        bal = est.results()
    finally:
        est.close()
    assert res["t_iter"][0] <= bal["t_iter"][0]


def test_pruning_is_exact():
    w = wl.make("small")
    _say(f"small: {w.n_cells} cells with and without bound pruning")
    a, ca, size = _run(w, prune=True)
    b, cb, _ = _run(w, prune=False)
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(a[k], b[k]), k
    assert ca["plans"] + ca["plans_skipped"] == size["plans"] and cb["plans_skipped"] == 0
    _say(f"  pruned: {ca['mem_partitions']} exact-T solves; exhaustive: {cb['mem_partitions']}")
    assert ca["mem_partitions"] < cb["mem_partitions"]


def test_never_slower_than_the_memory_rule():
    w = wl.make("trace")
    _say("trace: exact-T against the memory rule on every cell")
    a, _, _ = _run(w, with_cuts=False)
    est = arena.Estimator(w, rule=arena.PARTITION_MEMORY)
    try:
        est.estimate()
        m = est.results()
    finally:
        est.close()
    fin = np.isfinite(m["t_iter"])
    assert (np.isfinite(a["t_iter"]) == fin).all()
    assert (a["t_iter"][fin] <= m["t_iter"][fin] * (1 + 1e-6)).all()
    _say(f"  faster than the memory rule on {int((a['t_iter'][fin] < m['t_iter'][fin] * (1 - 1e-6)).sum())} "
         f"of {int(fin.sum())} feasible cells")


def test_refused_beyond_its_layer_limit():
    w = wl.make("moe")          # 128 layers per job
    est = arena.Estimator(w, rule=RULE)
    try:
        with pytest.raises(arena.ArenaError) as ei:
            est.estimate()
        assert ei.value.status == arena.ARENA_ERR_UNSUPPORTED
    finally:
        est.close()
