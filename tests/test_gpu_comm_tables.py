"""Parity of the interpolated communication latency (arena_set_comm_tables)
with the CPU oracle's table model, through the C ABI.

Every plan gets the balanced partition of its own per-microbatch costs, with
each communication term's latency interpolated in its link's table.  Small
workloads are compared cell by cell, the large ones run in full on the GPU
and are compared on sampled cells.  Each case prints its name first."""
import dataclasses
import sys

import numpy as np
import pytest

from paper_2403_16125_amd import arena
from paper_2403_16125_amd import workloads as wl

from compare import compare

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[commtab]", *a, flush=True)
    sys.stdout.flush()


def _run(w, tables, ids=None, with_cuts=True, prune=True):
    est = arena.Estimator(w, with_cuts=with_cuts, comm_tables=tables, prune=prune)
    try:
        est.estimate()
        res = est.results(ids)
        cnt = est.counters()
        size = est.space_size()
    finally:
        est.close()
    return res, cnt, size


def _check(rep, name, max_near_tie_frac=1e-3):
    _say(f"{name}: n={rep['n']} exact={rep['exact']} near_tie={rep['near_tie']} "
         f"mismatch={len(rep['mismatch'])} infeasible={rep['infeasible']} max_rel_T={rep['max_rel_T']:.3g}")
    assert not rep["mismatch"], rep["mismatch"][:5]
    assert rep["near_tie"] <= max(2, max_near_tie_frac * rep["n"])


def _sample(w, k, seed, whole_jobs=1):
    rng = np.random.default_rng(seed)
    ids = set(rng.choice(w.n_cells, size=min(k, w.n_cells), replace=False).tolist())
    per_job = w.n_types * w.n_counts
    for j in rng.choice(w.n_jobs, size=whole_jobs, replace=False):
        ids.update(range(int(j) * per_job, (int(j) + 1) * per_job))
    return np.asarray(sorted(ids), np.int64)


def test_hand_cell():
    """The oracle's hand cell: tables (0, 0.25 s), (5e8 B, 0.65 s), (1e9 B, 1.25 s)
    on both links; the cell's best plan is (2, 1, 1, 1) at T = 1.65 among 5."""
    _say("hand cell")
    job = dict(t=[1.0, 1.0], p=[2.5e8, 2.5e8], a=[0.0, 0.0], x=[5e8, 5e8], a2a=[0.0, 0.0], batch=2)
    ty = dict(speed=1.0, mem=1e15, bw_intra=1e9, bw_inter=1e9, gpus_per_node=2)
    w = wl.from_lists([job], [ty], [2], [1, 2], kappa=1.0)
    vol = np.broadcast_to(np.array([0.0, 5e8, 1e9]), (1, 2, 3)).copy()
    lat = np.broadcast_to(np.array([0.25, 0.65, 1.25]), (1, 2, 3)).copy()
    res, cnt, _ = _run(w, (vol, lat))
    assert (res["dp"][0], res["tp"][0], res["pp"][0], res["m"][0]) == (2, 1, 1, 1)
    assert res["t_iter"][0] == pytest.approx(1.65, rel=1e-6) and cnt["plans"] + cnt["plans_skipped"] == 5


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_every_cell(oracle, name):
    w = wl.make(name)
    tabs = wl.comm_tables(w)
    _say(f"{name}: {w.n_cells} cells, all compared")
    res, cnt, size = _run(w, tabs)
    _check(compare(w, res, np.arange(w.n_cells), oracle, tables=tabs), name)
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]


@pytest.mark.parametrize("name,k", [("trace", 400), ("moe", 150)])
def test_full_size_sampled(oracle, name, k):
    w = wl.make(name)
    tabs = wl.comm_tables(w)
    ids = _sample(w, k, seed=41)
    _say(f"{name}: {w.n_cells} cells on the GPU, {len(ids)} compared")
    res, cnt, size = _run(w, tabs, ids=ids)
    _check(compare(w, res, ids, oracle, tables=tabs), name)
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]


def test_full_round_sampled(oracle):
    w = wl.full()
    tabs = wl.comm_tables(w)
    ids = _sample(w, 300, seed=43)
    _say(f"full round: {w.n_cells} cells on the GPU, {len(ids)} compared")
    res, cnt, size = _run(w, tabs, ids=ids)
    _check(compare(w, res, ids, oracle, tables=tabs), "full")
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]


def test_edge_cases(oracle):
    sys.path.insert(0, __file__.rsplit("/", 1)[0])
    from test_gpu_parity import _edge_workload
    w = _edge_workload()
    tabs = wl.comm_tables(w)
    _say(f"edge: {w.n_cells} cells, all compared")
    res, _, _ = _run(w, tabs)
    rep = compare(w, res, np.arange(w.n_cells), oracle, tables=tabs)
    _check(rep, "edge")
    assert rep["infeasible"] > 0 and res["pp"].max() >= 64


def test_linear_tables_match_the_bandwidth_model():
    """Tables linear through the origin give the volume / bandwidth estimate:
    the same plans and cuts, T within f32 rounding, on every cell of small."""
    w = wl.make("small")
    _say("linear tables vs bandwidth model: small")
    r0, _, _ = _run(w, None)
    r1, _, _ = _run(w, wl.linear_tables(w, K=3))
    same = (r0["plan"] == r1["plan"]) & np.all(r0["cuts"] == r1["cuts"], axis=1)
    assert same.mean() >= 0.999, same.mean()
    fin = np.isfinite(r0["t_iter"])
    assert np.array_equal(fin, np.isfinite(r1["t_iter"]))
    rel = np.abs(r1["t_iter"][fin & same] - r0["t_iter"][fin & same]) / r0["t_iter"][fin & same]
    assert rel.max() <= 1e-6


def test_tables_switch_on_one_context():
    w = wl.full(n_jobs=24, rounds=1)
    tabs = wl.comm_tables(w)
    _say("tables on and off on one context: full[24 jobs]")
    ra, _, _ = _run(w, None)
    rb, _, _ = _run(w, tabs)
    est = arena.Estimator(w, with_cuts=True)
    try:
        est.set_comm_tables(tabs)
        est.estimate()
        x1 = est.results()
        est.set_comm_tables(None)
        est.estimate()
        x0 = est.results()
    finally:
        est.close()
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(x1[k], rb[k]), k
        assert np.array_equal(x0[k], ra[k]), k


@pytest.mark.parametrize("name", ["trace", "moe"])
def test_bound_pruning_is_exact(name):
    """Pruning plans whose lower bound lies past the tie window changes nothing:
    the whole launch bitwise equal with pruning off."""
    w = wl.make(name)
    tabs = wl.comm_tables(w)
    _say(f"{name}: tables with pruning on and off")
    r1, c1, size = _run(w, tabs)
    r0, c0, _ = _run(w, tabs, prune=False)
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(r1[k], r0[k]), k
    assert c0["plans_skipped"] == 0 and c0["plans"] == size["plans"]
    assert c1["plans"] + c1["plans_skipped"] == size["plans"] and c1["plans_skipped"] > 0
    _say(f"{name}: {c1['plans_skipped']} of {size['plans']} plans skipped")


def test_shared_bottlenecks_are_exact():
    """With one kappa for all counts of a type, cells of a (job, type) share the
    bottlenecks of their (tp, microbatch size) groups.  Raising the kappa of one
    count by one ulp turns the sharing off for that type: every other cell must
    come out bitwise the same, with fewer recursions when shared."""
    w = wl.moe(n_jobs=256)
    tabs = wl.comm_tables(w)
    k2 = w.kappa.copy()
    last = np.arange(w.n_types) * w.n_counts + (w.n_counts - 1)
    k2[:, last] = np.nextafter(k2[:, last], np.float32(2.0))
    w2 = dataclasses.replace(w, kappa=k2)
    _say(f"moe[256 jobs]: {w.n_cells} cells, kappa uniform vs one count off by an ulp")
    r1, c1, _ = _run(w, tabs)
    r2, c2, _ = _run(w2, tabs)
    keep = np.ones(w.n_cells, bool)
    keep[(np.arange(w.n_cells) % w.n_counts) == w.n_counts - 1] = False
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(r1[k][keep], r2[k][keep]), k
    _say(f"  recursions {c1['problems']} shared, {c2['problems']} unshared")
    assert c1["problems"] < c2["problems"]
