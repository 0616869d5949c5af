"""Pins of the oracle's plan pricing and per-cell choice (CPU only).

Fixed outside the oracle:
  * hand-derived cells (tests/golden/cells_hand.json), each term worked out
    by hand from the 1F1B model of Sec. 3.4 and the comm terms of Eq. 4;
  * closed forms: one GPU runs the whole model, so T is the sum of the layer
    times on that GPU whatever the microbatch count; with free communication
    and no pipeline, data parallelism scales linearly (the linear law the
    paper attributes to Sia, Sec. 2.3 strawman) and only there;
  * exact power-of-two rescaling of time and bandwidth units;
  * monotonicity that follows from the model (memory only removes plans,
    contention only slows comm, bandwidth only speeds it);
  * directional plan preferences the paper reports (Sec. 2.2: ample resources
    favour DP, tight memory favours MP/PP, slow links favour PP);
  * an independent enumeration of the plan space on small cells.
"""
import json
import math
import os

import numpy as np
import pytest

from paper_2403_16125_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = json.load(open(os.path.join(HERE, "golden", "cells_hand.json")))


def _one_cell(case, mem=None):
    ty = dict(case["type"])
    if mem is not None:
        ty["mem"] = mem
    return wl.from_lists([case["job"]], [ty], [case["n"]], case["m_values"],
                         kappa=case["kappa"])


@pytest.mark.parametrize("case", GOLDEN["cases"], ids=[c["name"] for c in GOLDEN["cases"]])
def test_golden_plans(oracle, case):
    w = _one_cell(case)
    for pl in case["plans"]:
        r = oracle.eval_plan(w, 0, 0, case["n"], case["kappa"], pl["dp"], pl["tp"], pl["pp"], pl["m"])
        assert r["T"] == pytest.approx(pl["T"], rel=1e-12), pl
        assert r["mem_max"] == pytest.approx(pl["mem_max"], rel=1e-12), pl
        if "cuts" in pl:
            assert r["cuts"] == pl["cuts"]


@pytest.mark.parametrize("case", GOLDEN["cases"], ids=[c["name"] for c in GOLDEN["cases"]])
def test_golden_best(oracle, case):
    if "best" not in case:
        pytest.skip("plan-level case only")
    w = _one_cell(case)
    r = oracle.cells(w, [0])
    b = case["best"]
    assert (r["dp"][0], r["tp"][0], r["pp"][0], r["m"][0]) == (b["dp"], b["tp"], b["pp"], b["m"])
    assert r["T"][0] == pytest.approx(b["T"], rel=1e-12)
    assert r["thr"][0] == pytest.approx(b["thr"], rel=1e-12)
    assert r["nplans"][0] == len(case["plans"])
    for v in case.get("variants", []):
        rv = oracle.cells(_one_cell(case, mem=v["mem"]), [0])
        if v["best"] is None:
            assert math.isinf(rv["T"][0]) and rv["thr"][0] == 0.0 and rv["dp"][0] == 0
            assert (rv["cuts"][0] == -1).all()
        else:
            vb = v["best"]
            assert (rv["dp"][0], rv["tp"][0], rv["pp"][0], rv["m"][0]) == \
                (vb["dp"], vb["tp"], vb["pp"], vb["m"])
            assert rv["T"][0] == pytest.approx(vb["T"], rel=1e-12)


def _cells_with_count(w, n):
    ci = int(np.nonzero(w.counts == n)[0][0])
    return np.asarray([(j * w.n_types + g) * w.n_counts + ci
                       for j in range(w.n_jobs) for g in range(w.n_types)], np.int64)


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_single_gpu_is_sum_of_layer_times(oracle, name):
    """n = 1: the whole model on one GPU; T = sum_l t_l / speed for every m, so
    the tie rule picks the smallest microbatch count whose activations fit."""
    w = wl.make(name)
    ids = _cells_with_count(w, 1)
    r = oracle.cells(w, ids)
    for s, c in enumerate(ids):
        j, g = int(c // (w.n_types * w.n_counts)), int((c // w.n_counts) % w.n_types)
        t = w.t[w.job_slice(j)].astype(np.float64)
        if np.isinf(r["T"][s]):
            continue            # too big for one GPU of this type
        assert r["T"][s] == pytest.approx(t.sum() / float(w.speed[g]), rel=1e-12)
        assert (r["dp"][s], r["tp"][s], r["pp"][s]) == (1, 1, 1)
        fits = [int(m) for m in w.m_values if w.batch[j] % m == 0 and
                oracle.eval_plan(w, j, g, 1, 1.0, 1, 1, 1, int(m))["feasible"]]
        assert r["m"][s] == min(fits)
    assert np.isfinite(r["T"]).sum() >= len(ids) // 2


def test_linear_scaling_only_without_communication(oracle):
    base = wl.small()
    inf = np.float32(np.inf)
    free = wl.Workload(**{**base.__dict__, "bw_intra": np.full(3, inf, np.float32),
                          "bw_inter": np.full(3, inf, np.float32),
                          "mem": np.full(3, 1e15, np.float32)})
    for j in range(0, base.n_jobs, 7):
        bg = int(base.batch[j])
        thr1 = bg / oracle.eval_plan(free, j, 0, 1, 1.0, 1, 1, 1, 1)["T"]
        for k in (2, 4, 8, 16, 32, 64):
            if bg % k:
                continue
            tk = oracle.eval_plan(free, j, 0, k, 1.0, k, 1, 1, 1)["T"]
            assert bg / tk == pytest.approx(k * thr1, rel=1e-12)
            # with a finite link the gradient all-reduce breaks the linear law
            tk_real = oracle.eval_plan(base, j, 0, k, 1.0, k, 1, 1, 1)["T"]
            assert bg / tk_real < k * thr1 * (1 - 1e-6)


@pytest.mark.parametrize("e", [3, -2, 10])
def test_power_of_two_rescaling_is_exact(oracle, e):
    """Seconds scaled by 2^e and bandwidths by 2^-e: every iteration time scales
    by exactly 2^e and every plan and cut is unchanged."""
    w = wl.trace(n_jobs=12)
    s = np.float32(2.0 ** e)
    w2 = wl.Workload(**{**w.__dict__, "t": w.t * s, "bw_intra": w.bw_intra / s,
                        "bw_inter": w.bw_inter / s})
    ids = np.arange(0, w.n_cells, 3, dtype=np.int64)
    r1, r2 = oracle.cells(w, ids), oracle.cells(w2, ids)
    fin = np.isfinite(r1["T"])
    assert fin.sum() > len(ids) // 2
    assert np.array_equal(r1["T"][fin] * 2.0 ** e, r2["T"][fin])
    assert np.array_equal(np.isinf(r1["T"]), np.isinf(r2["T"]))
    for k in ("dp", "tp", "pp", "m", "cuts"):
        assert np.array_equal(r1[k], r2[k])


def test_more_memory_never_hurts(oracle):
    w = wl.trace(n_jobs=16)
    w2 = wl.Workload(**{**w.__dict__, "mem": w.mem * np.float32(1.5)})
    ids = np.arange(w.n_cells, dtype=np.int64)
    r1, r2 = oracle.cells(w, ids), oracle.cells(w2, ids)
    assert (r2["T"] <= r1["T"] * (1 + w.tie_eps)).all()
    assert np.isfinite(r2["T"]).sum() >= np.isfinite(r1["T"]).sum()
    assert (r2["T"] < r1["T"]).any()


def test_bottleneck_monotone_in_kappa_and_bandwidth(oracle):
    w = wl.moe(n_jobs=6)
    for j in range(w.n_jobs):
        for tp in (2, 4, 8):
            for pp in (2, 8, 32):
                def wstar(kappa, scale=1.0):
                    ww = wl.Workload(**{**w.__dict__, "bw_intra": w.bw_intra * np.float32(scale),
                                        "bw_inter": w.bw_inter * np.float32(scale)})
                    u = oracle.layer_costs(ww, j, 2, kappa, 2, tp)
                    return oracle.bottleneck_dp(oracle.prefix(u), pp)
                w1, w2, w3 = wstar(1.0), wstar(1.7), wstar(1.0, 4.0)
                assert w2 >= w1 * (1 - 1e-12) and w2 > w1
                assert w3 <= w1 * (1 + 1e-12) and w3 < w1


def _best(oracle, w, n):
    r = oracle.cells(w, [int(np.nonzero(w.counts == n)[0][0])])
    return {k: int(r[k][0]) for k in ("dp", "tp", "pp", "m")}, r["T"][0]


def _one_type(speed=1.0, mem=80e9, bwi=300e9, bwe=25e9, gpn=8):
    return dict(speed=speed, mem=mem, bw_intra=bwi, bw_inter=bwe, gpus_per_node=gpn)


def _gpt_job(L=24, params=1.3e9, batch=256):
    pi = params / L
    h = 64 * round(math.sqrt(pi / 12) / 64)
    t = [6 * pi * batch * 1024 / 1e14] * L
    a = [64.0 * 1024 * h] * L
    return dict(t=t, p=[4 * pi] * L, a=a, x=[v / 16 for v in a], a2a=[0.0] * L, batch=batch)


def test_ample_resources_prefer_data_parallelism(oracle):
    job = _gpt_job(params=0.3e9)
    w = wl.from_lists([job], [_one_type(mem=1e13, bwi=1e13, bwe=1e13)], [8], [1, 2, 4, 8, 16])
    plan, _ = _best(oracle, w, 8)
    assert plan["dp"] == 8


def test_tight_memory_prefers_model_or_pipeline_parallelism(oracle):
    job = _gpt_job(params=6.7e9)
    ample = wl.from_lists([job], [_one_type(mem=1e13)], [8], [1, 2, 4, 8, 16, 32])
    tight = wl.from_lists([job], [_one_type(mem=40e9)], [8], [1, 2, 4, 8, 16, 32])
    p_ample, t_ample = _best(oracle, ample, 8)
    p_tight, t_tight = _best(oracle, tight, 8)
    assert p_tight["tp"] * p_tight["pp"] > p_ample["tp"] * p_ample["pp"]
    assert t_tight >= t_ample


def test_slow_links_prefer_pipeline_parallelism(oracle):
    job = _gpt_job(params=2.6e9, L=32)
    # one GPU per node: no tensor parallelism; DP pays a gradient all-reduce
    # over the inter-node link, PP only ships activations
    fast = wl.from_lists([job], [_one_type(mem=1e13, bwe=1e13, gpn=1)], [8], [1, 2, 4, 8, 16, 32])
    slow = wl.from_lists([job], [_one_type(mem=1e13, bwe=1e9, gpn=1)], [8], [1, 2, 4, 8, 16, 32])
    p_fast, _ = _best(oracle, fast, 8)
    p_slow, _ = _best(oracle, slow, 8)
    assert p_fast["pp"] == 1
    assert p_slow["pp"] > 1


def _enumerate(n, G, L, Bg, ms):
    out = []
    for tp in range(1, n + 1):
        if n % tp or tp > G or G % tp:
            continue
        for pp in range(1, n // tp + 1):
            if (n // tp) % pp or pp > L:
                continue
            dp = n // (tp * pp)
            out += [(dp, tp, pp, m) for m in ms if Bg % (dp * m) == 0]
    return out


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_enumeration_and_choice(oracle, name):
    """Independent re-enumeration of every plan of a cell and the tie rule."""
    w = wl.make(name)
    rng = np.random.default_rng(5)
    ids = rng.choice(w.n_cells, size=min(w.n_cells, 120), replace=False).astype(np.int64)
    r = oracle.cells(w, ids)
    for s, c in enumerate(ids):
        ci = int(c % w.n_counts)
        g = int((c // w.n_counts) % w.n_types)
        j = int(c // (w.n_counts * w.n_types))
        n = int(w.counts[ci])
        plans = _enumerate(n, int(w.gpus_per_node[g]), w.layers(j), int(w.batch[j]),
                           [int(m) for m in w.m_values])
        assert r["nplans"][s] == len(plans)
        kap = float(w.kappa[0][g * w.n_counts + ci])
        priced = []
        for (dp, tp, pp, m) in plans:
            e = oracle.eval_plan(w, j, g, n, kap, dp, tp, pp, m)
            if e["feasible"]:
                priced.append((e["T"], (pp, tp, m), (dp, tp, pp, m)))
        if not priced:
            assert np.isinf(r["T"][s])
            continue
        tmin = min(p[0] for p in priced)
        cand = sorted((p for p in priced if p[0] <= tmin * (1 + w.tie_eps)), key=lambda p: p[1])
        assert (r["dp"][s], r["tp"][s], r["pp"][s], r["m"][s]) == cand[0][2]
        assert r["T"][s] == cand[0][0]


# ---------------------------------------------------------------- hand-derived tie-breaks and links

def _cell(job, ty, n, m_values, tie_eps=1e-6):
    return wl.from_lists([job], [ty], [n], m_values, kappa=1.0, tie_eps=tie_eps)


@pytest.mark.parametrize("tie_eps", [1e-6, 0.0])
def test_tie_prefers_fewer_stages_then_less_tp(oracle, tie_eps):
    """Two layers of time 1 (whole batch of 2), boundary activations x = [0, 1/16],
    weights 0 and 10 bytes, 2 GPUs on one node of 2, links of 1 byte/s, m in {1, 2}.
      (dp, tp, pp) = (1, 2, 1): u_l = 1/(2*2) + 8 (1/2) x_l = 0.25, 0.5; T = Bg sum u
        = 2 x 0.75 = 1.5 for m = 1 and m = 2 (b = 2/m, m b = 2);
      (1, 1, 2): u = 0.5, 0.5, cuts [1], p2p carries x_0 = 0: m = 2 gives
        (0.5 + 0.5) + (2 - 1) x 0.5 = 1.5, m = 1 gives 2;
      (2, 1, 1): T = 1 + all-reduce 2 (1/2) 10 / 1 = 11 (m = 1 only).
    Three plans tie at exactly 1.5; the key (pp, tp, m) picks (1, 2, 1) over
    (pp 2, tp 1).  With a zero tie tolerance the best plan itself still counts."""
    job = dict(t=[1.0, 1.0], p=[0.0, 10.0], a=[0.0, 0.0], x=[0.0, 0.0625], a2a=[0.0, 0.0], batch=2)
    ty = dict(speed=1.0, mem=1e12, bw_intra=1.0, bw_inter=1.0, gpus_per_node=2)
    r = oracle.cells(_cell(job, ty, 2, [1, 2], tie_eps), [0])
    assert (r["dp"][0], r["tp"][0], r["pp"][0], r["m"][0]) == (1, 2, 1, 1)
    assert r["T"][0] == 1.5
    w = _cell(job, ty, 2, [1, 2], tie_eps)
    assert oracle.eval_plan(w, 0, 0, 2, 1.0, 1, 1, 2, 2)["T"] == 1.5
    assert oracle.eval_plan(w, 0, 0, 2, 1.0, 2, 1, 1, 1)["T"] == 11.0


def test_p2p_carries_the_last_layer_of_the_stage(oracle):
    """Two layers of time 1 (batch 1), x = [0.5, 0.25], 2 GPUs on one node of 2,
    links of 1 byte/s; plan (1, 1, 2, 1): b = 1, stages [0,1) [1,2) of time 1 each,
    the boundary after layer 0 carries 2 x 1 x x_0 = 1 (activation out, gradient
    back): T = (1 + 1) + 1 = 3."""
    job = dict(t=[1.0, 1.0], p=[0.0, 0.0], a=[0.0, 0.0], x=[0.5, 0.25], a2a=[0.0, 0.0], batch=1)
    ty = dict(speed=1.0, mem=1e12, bw_intra=1.0, bw_inter=1.0, gpus_per_node=2)
    e = oracle.eval_plan(_cell(job, ty, 2, [1]), 0, 0, 2, 1.0, 1, 1, 2, 1)
    assert e["cuts"] == [1] and e["T"] == 3.0


def test_dp_group_not_dividing_the_node_uses_the_inter_node_link(oracle):
    """One layer of time 3 (batch 3), 3e9 bytes of weights, nodes of 4 GPUs,
    intra 1e10 and inter 1e9 bytes/s; plan (3, 1, 1, 1): b = 1, compute 3/3 = 1;
    the dp group of 3 fits a node but does not divide it, so its gradient
    all-reduce 2 (2/3) 3e9 crosses the inter-node link: 4 s; T = 5."""
    job = dict(t=[3.0], p=[3e9], a=[0.0], x=[0.0], a2a=[0.0], batch=3)
    ty = dict(speed=1.0, mem=1e12, bw_intra=1e10, bw_inter=1e9, gpus_per_node=4)
    e = oracle.eval_plan(_cell(job, ty, 3, [1]), 0, 0, 3, 1.0, 3, 1, 1, 1)
    assert e["T"] == pytest.approx(5.0, rel=1e-15)
