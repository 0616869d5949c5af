"""Parity of the memory-constrained partition rule (ARENA_PARTITION_MEMORY)
with the CPU oracle's rule 1, through the C ABI.

Under the rule a plan's stages are the balanced partition (Sec. 3.2) among
the splits whose every stage fits memory (Sec. 3.3).  Small workloads are
compared cell by cell, the large ones run in full and are compared on sampled
cells; the rule is also checked against the balanced rule on the same
launches (no cell slower, every balanced-feasible cell still feasible) and
with bound pruning off (identical outputs).  Each case prints its name first.
"""
import sys

import numpy as np
import pytest

from paper_2403_16125_amd import arena
from paper_2403_16125_amd import workloads as wl

from compare import compare

pytestmark = pytest.mark.gpu
MEM = arena.PARTITION_MEMORY


def _say(*a):
    print("[memrule]", *a, flush=True)
    sys.stdout.flush()


def _run(w, rule=MEM, rnd=0, with_cuts=True, ids=None, prune=True):
    est = arena.Estimator(w, with_cuts=with_cuts, prune=prune, rule=rule)
    try:
        if rnd:
            est.set_round(rnd)
        est.estimate()
        res = est.results(ids)
        cnt = est.counters()
        size = est.space_size()
    finally:
        est.close()
    return res, cnt, size


def _check(rep, name, max_near_tie_frac=1e-3):
    _say(f"{name}: n={rep['n']} exact={rep['exact']} near_tie={rep['near_tie']} "
         f"mismatch={len(rep['mismatch'])} infeasible={rep['infeasible']} "
         f"max_rel_T={rep['max_rel_T']:.3g}")
    assert not rep["mismatch"], rep["mismatch"][:5]
    assert rep["near_tie"] <= max(2, max_near_tie_frac * rep["n"])


def _sample(w, k, seed, whole_jobs=2):
    rng = np.random.default_rng(seed)
    ids = set(rng.choice(w.n_cells, size=min(k, w.n_cells), replace=False).tolist())
    per_job = w.n_types * w.n_counts
    for j in rng.choice(w.n_jobs, size=whole_jobs, replace=False):
        ids.update(range(int(j) * per_job, (int(j) + 1) * per_job))
    return np.asarray(sorted(ids), np.int64)


def test_hand_cells():
    """The two hand-derived cells of the oracle's pins: infeasible under the
    balanced rule, T = 4 (cuts [1]) and T = 10 (cuts [1, 2]) under the rule."""
    _say("hand cells")
    job1 = dict(t=[1, 1, 1, 1], p=[3e9, 1e9, 1e9, 1e9], a=[0] * 4, x=[0] * 4, a2a=[0] * 4, batch=1)
    ty1 = dict(speed=1.0, mem=12e9, bw_intra=1e9, bw_inter=1e9, gpus_per_node=1)
    job2 = dict(t=[2, 2, 2, 6], p=[0] * 4, a=[1e9] * 4, x=[0] * 4, a2a=[0] * 4, batch=2)
    ty2 = dict(speed=1.0, mem=2e9, bw_intra=1e9, bw_inter=1e9, gpus_per_node=1)
    for job, ty, n, ms, want in ((job1, ty1, 2, [1], (1, 1, 2, 1, 4.0, [1])),
                                 (job2, ty2, 3, [2], (1, 1, 3, 2, 10.0, [1, 2]))):
        w = wl.from_lists([job], [ty], [n], ms, kappa=1.0)
        r0, _, _ = _run(w, rule=arena.PARTITION_BALANCED)
        assert not r0["feasible"][0] and np.isinf(r0["t_iter"][0])
        r1, cnt, _ = _run(w)
        assert (r1["dp"][0], r1["tp"][0], r1["pp"][0], r1["m"][0]) == want[:4]
        assert r1["t_iter"][0] == pytest.approx(want[4], rel=1e-7)
        pp = want[2]
        assert list(r1["cuts"][0][:pp - 1]) == want[5] and r1["cuts"][0][pp - 1] == 0xFF
        assert cnt["mem_partitions"] >= 1


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_every_cell(oracle, name):
    w = wl.make(name)
    _say(f"{name}: {w.n_cells} cells, all compared")
    res, cnt, size = _run(w)
    rep = compare(w, res, np.arange(w.n_cells), oracle, rule=1)
    _check(rep, name)
    assert cnt["cells"] == w.n_cells
    assert cnt["plans"] + cnt["plans_skipped"] == size["plans"]


@pytest.mark.parametrize("name,k", [("trace", 400), ("moe", 120)])
def test_full_size_sampled(oracle, name, k):
    w = wl.make(name)
    ids = _sample(w, k, seed=23)
    _say(f"{name}: {w.n_cells} cells on the GPU, {len(ids)} compared")
    res, cnt, size = _run(w, ids=ids)
    _check(compare(w, res, ids, oracle, rule=1), name)
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]
    assert cnt["mem_partitions"] > 0


def test_full_round_sampled(oracle):
    w = wl.full()
    ids = _sample(w, 500, seed=31, whole_jobs=1)
    _say(f"full round: {w.n_cells} cells on the GPU, {len(ids)} compared")
    res, cnt, size = _run(w, ids=ids)
    _check(compare(w, res, ids, oracle, rule=1), "full")
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]


def test_edge_cases(oracle):
    sys.path.insert(0, __file__.rsplit("/", 1)[0])
    from test_gpu_parity import _edge_workload
    w = _edge_workload()
    _say(f"edge: {w.n_cells} cells, all compared")
    res, cnt, size = _run(w)
    rep = compare(w, res, np.arange(w.n_cells), oracle, rule=1)
    _check(rep, "edge")
    assert rep["infeasible"] > 0 and res["pp"].max() >= 64


@pytest.mark.parametrize("name", ["trace", "moe"])
def test_rule_never_slower_and_pruning_exact(name):
    """On the whole launch: every cell feasible under the balanced rule stays
    feasible and gets no slower, some cells gain; pruning off gives bitwise
    the same outputs."""
    w = wl.make(name)
    _say(f"{name}: balanced vs memory rule, pruning on and off")
    r0, _, _ = _run(w, rule=arena.PARTITION_BALANCED, with_cuts=False)
    r1, c1, _ = _run(w, with_cuts=True)
    r1n, c1n, _ = _run(w, with_cuts=True, prune=False)
    f0 = r0["feasible"]
    assert r1["feasible"][f0].all()
    assert (r1["t_iter"][f0] <= r0["t_iter"][f0]).all()
    gained = int((r1["feasible"] & ~f0).sum()) + int((r1["t_iter"][f0] < r0["t_iter"][f0]).sum())
    _say(f"{name}: {gained} cells gain, {c1['mem_partitions']} rule partitions "
         f"({c1n['mem_partitions']} unpruned)")
    assert gained > 0
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(r1[k], r1n[k]), k
    assert c1n["plans_skipped"] == 0 and c1["mem_partitions"] <= c1n["mem_partitions"]


def test_rule_switch_on_one_context():
    """Switching the rule on a live context gives each rule's fresh-context answer."""
    w = wl.full(n_jobs=48, rounds=2)
    _say("rule switch: full[48 jobs]")
    ra, _, _ = _run(w, rule=arena.PARTITION_BALANCED)
    rb, _, _ = _run(w, rule=MEM)
    est = arena.Estimator(w, with_cuts=True)
    try:
        est.set_partition_rule(MEM)
        est.estimate()
        x1 = est.results()
        est.set_partition_rule(arena.PARTITION_BALANCED)
        est.estimate()
        x0 = est.results()
    finally:
        est.close()
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(x1[k], rb[k]), k
        assert np.array_equal(x0[k], ra[k]), k
