"""Parity of the HIP estimator with the CPU oracle, through the C ABI.

Small workloads are compared cell by cell in full; the large ones run in full
on the GPU (the launch the benchmark times) and are compared on sampled cells
the oracle evaluates one by one.  Every case prints what it runs first, so a
failing run names its case.
"""
import json
import os
import sys

import numpy as np
import pytest

from paper_2403_16125_amd import arena
from paper_2403_16125_amd import workloads as wl

from compare import compare

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def _say(*a):
    print("[parity]", *a, flush=True)
    sys.stdout.flush()


def _run(w, rnd=0, with_cuts=True, ids=None):
    est = arena.Estimator(w, with_cuts=with_cuts)
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


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_every_cell(oracle, name):
    w = wl.make(name)
    _say(f"{name}: {w.n_cells} cells, all compared")
    res, cnt, size = _run(w)
    ids = np.arange(w.n_cells)
    rep = compare(w, res, ids, oracle)
    _check(rep, name)
    assert cnt["cells"] == w.n_cells
    # no plan is priced twice (the skipped count is the rest of the space)
    assert 0 < cnt["plans"] <= size["plans"]
    assert cnt["plans"] + cnt["plans_skipped"] == size["plans"]
    assert cnt["infeasible_cells"] == rep["infeasible"]


def _sample(w, k, seed, whole_jobs=2):
    rng = np.random.default_rng(seed)
    ids = set(rng.choice(w.n_cells, size=min(k, w.n_cells), replace=False).tolist())
    per_job = w.n_types * w.n_counts
    for j in rng.choice(w.n_jobs, size=whole_jobs, replace=False):
        ids.update(range(int(j) * per_job, (int(j) + 1) * per_job))
    return np.asarray(sorted(ids), np.int64)


@pytest.mark.parametrize("name,k", [("trace", 1500), ("moe", 300)])
def test_full_size_sampled(oracle, name, k):
    w = wl.make(name)
    ids = _sample(w, k, seed=11)
    _say(f"{name}: {w.n_cells} cells on the GPU, {len(ids)} compared")
    res, cnt, size = _run(w, ids=ids)
    _check(compare(w, res, ids, oracle), name)
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]


@pytest.mark.parametrize("rnd,with_cuts", [(0, True), (9, True), (4, False)])
def test_full_round_sampled(oracle, rnd, with_cuts):
    """The full round on the GPU, compared with the oracle on sampled cells.
    Without cut rows (4) this is exactly the launch the benchmark times (cut
    rows off, bound pruning on); the oracle then checks time and plan."""
    w = wl.full()
    ids = _sample(w, 1200, seed=100 + rnd, whole_jobs=1)
    _say(f"full round {rnd}, cut rows {'on' if with_cuts else 'off'}: {w.n_cells} cells on the GPU, "
         f"{len(ids)} compared")
    res, cnt, size = _run(w, rnd=rnd, with_cuts=with_cuts, ids=ids)
    assert ("cuts" in res) == with_cuts
    _check(compare(w, res, ids, oracle, kappa_round=rnd), f"full r{rnd}")
    assert cnt["cells"] == w.n_cells and cnt["plans"] + cnt["plans_skipped"] == size["plans"]


def test_full_round_timed_launch_bitwise_equals_cut_launch():
    """The benchmark's launch (no cut rows) writes, on every one of the 17.2 M
    cells of a full round, bitwise the times, throughputs and plans of the
    launch with cut rows, whose cells the oracle checks above."""
    import torch
    w = wl.full()
    _say(f"full round 6: {w.n_cells} cells with and without cut rows")
    out = []
    for with_cuts in (False, True):
        est = arena.Estimator(w, with_cuts=with_cuts)
        try:
            est.set_round(6)
            est.estimate()
            torch.cuda.synchronize()
            out.append((est.t_iter.clone(), est.thr.clone(), est.plan.clone()))
        finally:
            est.close()
    for k, (a, b) in zip(("t_iter", "thr", "plan"), zip(*out)):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32)), k


def _edge_workload():
    """Degenerate shapes: one layer, zero-cost layers, a dominant layer, the
    largest job (128 layers, pipeline degree up to 128), free links, cells
    that fit nowhere and counts with no plan at all."""
    rng = np.random.default_rng(3)
    jobs = []
    jobs.append(dict(t=[2e-3], p=[1e8], a=[1e6], x=[1e5], a2a=[0.0], batch=8))
    jobs.append(dict(t=[0.0, 1e-3, 0.0, 0.0, 2e-3], p=[1e8] * 5, a=[1e6] * 5, x=[1e5] * 5,
                     a2a=[0.0] * 5, batch=16))
    t = list(rng.uniform(1e-3, 2e-3, 40)); t[17] = 1.0
    jobs.append(dict(t=t, p=[5e7] * 40, a=[2e6] * 40, x=[1e5] * 40, a2a=[0.0] * 40, batch=64))
    L = 128
    jobs.append(dict(t=list(rng.lognormal(-6, 0.8, L)), p=list(rng.uniform(1e8, 3e8, L)),
                     a=[4e6] * L, x=[2.5e5] * L, a2a=[0.0 if i % 2 == 0 else 4e5 for i in range(L)],
                     batch=128))
    jobs.append(dict(t=[1e-3] * 24, p=[1e10] * 24, a=[1e9] * 24, x=[1e7] * 24, a2a=[0.0] * 24,
                     batch=4))                    # too big for most cells
    jobs.append(dict(t=[1.0] * 8, p=[1e8] * 8, a=[1e6] * 8, x=[1e5] * 8, a2a=[0.0] * 8,
                     batch=3))                    # odd batch: few admissible plans
    types = [dict(speed=1.0, mem=80e9, bw_intra=300e9, bw_inter=25e9, gpus_per_node=8),
             dict(speed=0.5, mem=16e9, bw_intra=np.inf, bw_inter=np.inf, gpus_per_node=1),
             dict(speed=0.7, mem=40e9, bw_intra=64e9, bw_inter=12.5e9, gpus_per_node=16)]
    counts = [1, 2, 3, 8, 24, 128, 256, 1024]
    kappa = rng.uniform(1.0, 2.0, len(types) * len(counts))
    return wl.from_lists(jobs, types, counts, [1, 2, 4, 8, 16, 32, 64], kappa=kappa)


def test_edge_cases(oracle):
    w = _edge_workload()
    _say(f"edge: {w.n_cells} cells, all compared")
    res, cnt, size = _run(w)
    rep = compare(w, res, np.arange(w.n_cells), oracle)
    _check(rep, "edge")
    assert rep["infeasible"] > 0 and rep["exact"] > rep["infeasible"]
    pp = res["pp"]
    assert pp.max() >= 64          # deep pipelines of the 128-layer job are exercised


GOLDEN = json.load(open(os.path.join(HERE, "golden", "cells_hand.json")))


@pytest.mark.parametrize("case", [c for c in GOLDEN["cases"] if "best" in c],
                         ids=[c["name"] for c in GOLDEN["cases"] if "best" in c])
def test_golden_cells(case):
    w = wl.from_lists([case["job"]], [case["type"]], [case["n"]], case["m_values"],
                      kappa=case["kappa"])
    _say(f"golden {case['name']}")
    res, _, _ = _run(w)
    b = case["best"]
    assert (res["dp"][0], res["tp"][0], res["pp"][0], res["m"][0]) == (b["dp"], b["tp"], b["pp"], b["m"])
    assert res["t_iter"][0] == pytest.approx(b["T"], rel=1e-6)
    assert res["thr"][0] == pytest.approx(b["thr"], rel=1e-6)


def test_bitwise_deterministic_and_permutation_equivariant():
    w = wl.trace(n_jobs=96)
    _say("determinism + permutation: trace[96 jobs]")
    r1, _, _ = _run(w)
    r2, _, _ = _run(w)
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(r1[k], r2[k]), k
    perm = np.random.default_rng(4).permutation(w.n_jobs)
    wp = w.subset_jobs(perm)
    rp, _, _ = _run(wp)
    per = w.n_types * w.n_counts
    rows = (perm[:, None] * per + np.arange(per)[None, :]).ravel()
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(rp[k], r1[k][rows]), k


def test_grid_permutation_equivariant():
    """Reordering the GPU types and the GPU counts of the grid (with their
    contention factors) only reorders the matrix: every cell, cut row
    included, is bitwise the same as the original cell it maps to."""
    import dataclasses
    w = wl.trace(n_jobs=64)
    _say("grid permutation: trace[64 jobs], 4 types x 35 counts permuted")
    r1, _, _ = _run(w)
    rng = np.random.default_rng(9)
    tperm = rng.permutation(w.n_types)
    cperm = rng.permutation(w.n_counts)
    kap = np.asarray(w.kappa).reshape(w.n_rounds, w.n_types, w.n_counts)[:, tperm][:, :, cperm]
    wp = dataclasses.replace(
        w, speed=w.speed[tperm].copy(), mem=w.mem[tperm].copy(), bw_intra=w.bw_intra[tperm].copy(),
        bw_inter=w.bw_inter[tperm].copy(), gpus_per_node=w.gpus_per_node[tperm].copy(),
        counts=w.counts[cperm].copy(), kappa=np.ascontiguousarray(kap.reshape(w.n_rounds, -1)),
        hbm=None if w.hbm is None else w.hbm[tperm].copy())
    rp, _, _ = _run(wp)
    # cell (j, g', c') of the permuted grid is cell (j, tperm[g'], cperm[c'])
    j = np.arange(w.n_jobs)[:, None, None]
    src = (j * w.n_types + tperm[None, :, None]) * w.n_counts + cperm[None, None, :]
    src = src.ravel()
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(rp[k], r1[k][src]), k


def test_no_cuts_and_kappa_rounds_consistent():
    """Without the cuts output the matrix is unchanged; changing kappa between
    rounds on one context gives the same answer as a fresh context."""
    w = wl.full(n_jobs=64, rounds=3)
    _say("cuts-free run and per-round kappa: full[64 jobs]")
    ra, _, _ = _run(w, rnd=2, with_cuts=True)
    rb, _, _ = _run(w, rnd=2, with_cuts=False)
    for k in ("t_iter", "thr", "plan"):
        assert np.array_equal(ra[k], rb[k]), k
    est = arena.Estimator(w, with_cuts=True)
    try:
        for r in (0, 1, 2):
            est.set_round(r)
            est.estimate()
        rc = est.results()
    finally:
        est.close()
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(ra[k], rc[k]), k


def test_invalid_device_values_are_rejected():
    import torch
    w = wl.tiny()
    w.t[5] = np.nan
    _say("invalid per-layer value")
    est = arena.Estimator(w, with_cuts=False)
    try:
        est.t_iter.fill_(7.0)
        with pytest.raises(arena.ArenaError) as ei:
            est.estimate()
        assert ei.value.status == arena.ARENA_ERR_INVALID_ARG
        torch.cuda.synchronize()
        assert (est.t_iter.cpu() == 7.0).all()      # nothing written
    finally:
        est.close()


def _both_modes(w, rnd, with_cuts):
    out = {}
    for prune in (True, False):
        est = arena.Estimator(w, with_cuts=with_cuts, prune=prune)
        try:
            if rnd:
                est.set_round(rnd)
            est.estimate()
            out[prune] = (est.results(), est.counters(), est.space_size())
        finally:
            est.close()
    return out


@pytest.mark.parametrize("name,rnd,with_cuts", [("full", 3, False), ("trace", 0, True), ("moe", 0, True)])
def test_bound_pruning_is_exact(name, rnd, with_cuts):
    """Bound pruning changes only the work: every cell (and every cut row) is
    bitwise identical with it on and off, and every plan is either priced or
    skipped."""
    w = wl.make(name)
    _say(f"{name} round {rnd}: {w.n_cells} cells with and without bound pruning")
    out = _both_modes(w, rnd, with_cuts)
    (a, ca, size), (b, cb, _) = out[True], out[False]
    keys = ("t_iter", "thr", "plan") + (("cuts",) if with_cuts else ())
    for k in keys:
        assert np.array_equal(a[k], b[k]), k
    _say(f"  pruned: {ca['plans']} plans priced, {ca['plans_skipped']} skipped, {ca['dp_entries']} entries; "
         f"exhaustive: {cb['plans']} plans, {cb['dp_entries']} entries")
    assert cb["plans_skipped"] == 0 and cb["plans"] == size["plans"]
    assert ca["plans"] + ca["plans_skipped"] == size["plans"]
    # shared problems (one contention factor per type) are solved whole either way
    assert ca["plans_skipped"] > 0 and ca["dp_entries"] <= cb["dp_entries"]
    assert ca["infeasible_cells"] == cb["infeasible_cells"]


def test_microbatch_order_irrelevant():
    """The plan space is a set: the order of the listed microbatch counts
    (sorted by the library for the kernel) does not change any result."""
    import dataclasses
    w = wl.make("small")
    w2 = dataclasses.replace(w, m_values=np.ascontiguousarray(w.m_values[::-1]))
    a, _, _ = _run(w)
    b, _, _ = _run(w2)
    for k in ("t_iter", "thr", "plan", "cuts"):
        assert np.array_equal(a[k], b[k]), k


def test_hand_tie_and_link_cells():
    """The hand-derived cells of the oracle's pins, through the HIP path: an exact
    three-way tie decided by the key (pp, tp, m) with tie tolerance 1e-6 and 0,
    the p2p of a stage boundary carrying the stage's last layer, and a data-
    parallel group that fits a node without dividing it (inter-node link)."""
    tie_job = dict(t=[1.0, 1.0], p=[0.0, 10.0], a=[0.0, 0.0], x=[0.0, 0.0625], a2a=[0.0, 0.0], batch=2)
    ty2 = dict(speed=1.0, mem=1e12, bw_intra=1.0, bw_inter=1.0, gpus_per_node=2)
    for eps in (1e-6, 0.0):
        _say(f"hand tie cell, tie_eps {eps}")
        w = wl.from_lists([tie_job], [ty2], [2], [1, 2], kappa=1.0, tie_eps=eps)
        res, _, _ = _run(w)
        assert (res["dp"][0], res["tp"][0], res["pp"][0], res["m"][0]) == (1, 2, 1, 1)
        assert res["t_iter"][0] == 1.5
    _say("hand p2p and dp-link cells")
    p2p_job = dict(t=[1.0, 1.0], p=[0.0, 0.0], a=[0.0, 0.0], x=[0.5, 0.25], a2a=[0.0, 0.0], batch=1)
    w = wl.from_lists([p2p_job], [ty2], [2], [1], kappa=1.0)
    res, _, _ = _run(w)
    # (1, 1, 2, 1) costs 3 (p2p 1 after layer 0); (1, 2, 1, 1) costs 1 + 4 x (0.5 + 0.25) = 4
    assert (res["dp"][0], res["tp"][0], res["pp"][0], res["m"][0]) == (1, 1, 2, 1)
    assert res["t_iter"][0] == 3.0 and list(res["cuts"][0][:2]) == [1, 0xFF]
    dp_job = dict(t=[3.0], p=[3e9], a=[0.0], x=[0.0], a2a=[0.0], batch=3)
    ty4 = dict(speed=1.0, mem=1e12, bw_intra=1e10, bw_inter=1e9, gpus_per_node=4)
    w = wl.from_lists([dp_job], [ty4], [3], [1], kappa=1.0)
    res, _, _ = _run(w)
    assert (res["dp"][0], res["tp"][0], res["pp"][0], res["m"][0]) == (3, 1, 1, 1)
    assert res["t_iter"][0] == pytest.approx(5.0, rel=1e-6)
