"""Pins of the proxy-plan oracle (CPU): the load-aware planner of Sec. 3.3
(roofline loads of Eq. 2, proportional GPU shares, the power-of-two
normalisation minimising the computation bias of Eq. 3, the communication
load of Eq. 4, the proxy choice) checked against brute force, closed forms,
the uniform-plan oracle and hand-derived cases."""
import itertools
import math

import numpy as np
import pytest

from oracle import oracle as uo
from oracle import proxy as px
from paper_2403_16125_amd import workloads as wl

F_REF = 1e14


def _pow2_vectors(s, n):
    pw = [1 << e for e in range(n.bit_length())]
    for v in itertools.product(pw, repeat=s):
        if sum(v) == n:
            yield v


@pytest.mark.parametrize("seed", range(60))
def test_normalisation_is_the_brute_force_minimum(seed):
    # every ordered vector of powers of two summing to n (no sorting, no
    # pairing argument) against the oracle's multiset search
    rng = np.random.default_rng(seed)
    s = int(rng.integers(1, 6))
    n = int(rng.choice([1, 2, 3, 4, 5, 6, 8, 12, 16, 24]))
    D = rng.dirichlet(np.ones(s)) * n
    if seed % 4 == 0 and s >= 2:
        D[s - 1] = D[0]                      # exact equal shares
    b2, m = px.normalize(D, n)
    vecs = list(_pow2_vectors(s, n))
    if not vecs:
        assert b2 is None
        return
    costs = [sum((v[j] - D[j]) ** 2 for j in range(s)) for v in vecs]
    best = min(costs)
    assert b2 == pytest.approx(best, rel=1e-12, abs=1e-12)
    assert sum(m) == n and all(x > 0 and x & (x - 1) == 0 for x in m)
    assert sum((m[j] - D[j]) ** 2 for j in range(s)) == pytest.approx(best, rel=1e-12, abs=1e-12)


def test_normalisation_special_cases():
    assert px.normalize([1.5], 3) == (None, None)            # 3 is no power of two
    assert px.normalize([1.0, 1.0, 1.0], 2) == (None, None)  # more stages than GPUs
    b2, m = px.normalize([4.0, 2.0, 2.0], 8)                 # already powers of two
    assert b2 == 0.0 and list(m) == [4, 2, 2]
    b2, m = px.normalize([12.0, 12.0], 24)                   # equal shares: the earlier stage
    assert b2 == 32.0 and list(m) == [16, 8]                 # gets the larger count
    b2, m = px.normalize([3.2, 0.8], 4)                      # (2-3.2)^2 + (2-0.8)^2
    assert b2 == pytest.approx(2.88, rel=1e-15) and list(m) == [2, 2]


def _one_type(speed=1.0, mem=80e9, bwi=300e9, bwe=25e9, gpn=8, hbm=2e12):
    return dict(speed=speed, mem=mem, bw_intra=bwi, bw_inter=bwe, gpus_per_node=gpn), hbm


def _workload(layers, batch, counts, m_values, **ty):
    t, hbm = _one_type(**ty)
    w = wl.from_lists([dict(batch=batch, **layers)], [t], counts, m_values)
    w.hbm = np.asarray([hbm], np.float32)
    return w


def _layers(L, t=1e-3, p=1e8, a=1e6, x=None, a2a=0.0):
    vals = lambda v: list(np.broadcast_to(np.asarray(v, np.float64), (L,)))
    return dict(t=vals(t), p=vals(p), a=vals(a), x=vals(np.asarray(a) / 16 if x is None else x),
                a2a=vals(a2a))


def test_operator_clusters_and_compute_bound_loads():
    # 40 layers of equal cost in 16 operators: floor(16 i / 40) boundaries give
    # operators of 2 or 3 layers; compute-bound load = layers x t / speed
    w = _workload(_layers(40, t=2e-3, p=1.0, a=1.0), 64, [8], [1], speed=0.5, hbm=1e30)
    load, d = px.loads(w, 0, 0, 8, F_REF)
    sizes = np.diff([(i * 40) // 16 for i in range(17)])
    assert len(load) == 16
    t32 = float(np.float32(2e-3))                           # the tables are f32
    np.testing.assert_allclose(load, sizes * t32 / 0.5, rtol=1e-12)
    assert d.sum() == pytest.approx(8.0, rel=1e-12)
    np.testing.assert_allclose(d, sizes / 40 * 8, rtol=1e-12)
    # fewer layers than operators: one layer each
    w = _workload(_layers(5, t=[1e-3, 2e-3, 3e-3, 4e-3, 5e-3], p=1.0, a=1.0), 64, [4], [1], hbm=1e30)
    load, d = px.loads(w, 0, 0, 4, F_REF)
    t32 = np.array([1e-3, 2e-3, 3e-3, 4e-3, 5e-3], np.float32).astype(np.float64)
    np.testing.assert_allclose(load, t32, rtol=1e-12)
    np.testing.assert_allclose(d, t32 / t32.sum() * 4, rtol=1e-12)


def test_memory_bound_loads():
    # a tiny memory bandwidth makes every operator memory-bound: load = (p + Bg a) / bandwidth
    w = _workload(_layers(4, t=1e-9, p=[1e6, 2e6, 3e6, 4e6], a=[1e3, 1e3, 2e3, 2e3]), 32, [4], [1],
                  hbm=1e3)
    load, d = px.loads(w, 0, 0, 4, F_REF)
    want = (np.array([1e6, 2e6, 3e6, 4e6]) + 32 * np.array([1e3, 1e3, 2e3, 2e3])) / 1e3
    np.testing.assert_allclose(load, want, rtol=1e-6)      # f32 inputs
    np.testing.assert_allclose(d, want / want.sum() * 4, rtol=1e-6)


@pytest.mark.parametrize("plan", [
    # (n, s, dp, tp, B, cuts in layers = operators)
    (8, 2, 2, 2, 4, [7]), (8, 4, 2, 1, 8, [3, 9, 12]), (16, 2, 4, 2, 2, [8]), (4, 1, 2, 2, 4, []),
    (16, 8, 1, 2, 16, [1, 2, 5, 8, 9, 13, 15]), (8, 2, 1, 4, 1, [10]),
])
def test_uniform_plans_price_as_the_uniform_oracle(plan):
    # one layer per operator, every stage with the same (dp, tp): the per-stage
    # model must equal the uniform 1F1B oracle (same formulas, other sums)
    n, s, dp, tp, B, cuts = plan
    rng = np.random.default_rng(n * 100 + s)
    layers = dict(t=list(rng.uniform(1e-3, 5e-3, 16)), p=list(rng.uniform(5e7, 1.5e8, 16)),
                  a=list(rng.uniform(2e7, 6e7, 16) / 64), x=list(rng.uniform(1e5, 1e6, 16)),
                  a2a=list(np.where(np.arange(16) % 2 == 1, 4e5, 0.0)))
    w = _workload(layers, 64, [n], [B], mem=1e13, gpn=4)
    kap = 1.3
    bounds = [0] + cuts + [16]
    T, feas, _ = px.price(w, 0, 0, n, kap, bounds, [dp * tp] * s, [tp] * s, B, F_REF)
    ref = uo.eval_plan(w, 0, 0, n, kap, dp, tp, s, B, cuts=cuts)
    assert feas and ref["feasible"]
    assert T == pytest.approx(ref["T"], rel=1e-12)


def test_communication_load_by_hand():
    # 2 layers = 2 operators, 2 stages, B = 4, Bg = 64, kappa 1.5
    # stage 0: 4 GPUs as dp 2 x tp 2; stage 1: 2 GPUs as dp 2 x tp 1
    x = [1e6, 2e6]
    a2a = [3e5, 0.0]
    p = [8e8, 4e8]
    w = _workload(dict(t=[1e-3, 1e-3], p=p, a=[1e3, 1e3], x=x, a2a=a2a), 64, [6], [4],
                  bwi=100e9, bwe=10e9, gpn=4, mem=1e13)
    kap, B = 1.5, 4
    T, feas, lcomm = px.price(w, 0, 0, 6, kap, [0, 1, 2], [4, 2], [2, 1], B, F_REF)
    b0 = 64 / (2 * B)                  # samples per replica per microbatch, stage 0
    b1 = 64 / (2 * B)
    C0 = b0 * (kap * 8 * 1 / 2 * x[0] / 100e9 + kap * a2a[0] / 10e9)
    C1 = b1 * (kap * a2a[1] / 10e9)    # tp 1: no all-reduce; no all-to-all on the dense layer
    AR0 = kap * 2 * (2 - 1) / 2 * (p[0] / 2) / 100e9     # 4 GPUs divide the node of 4: intra
    AR1 = kap * 2 * (2 - 1) / 2 * (p[1] / 1) / 100e9     # 2 GPUs: intra
    want = (B - 1) * max(C0, C1) + (C0 + C1) + (AR0 + AR1)
    assert feas
    assert lcomm == pytest.approx(want, rel=1e-6)


def test_intra_stage_choice_follows_the_communication():
    # one stage of 8 GPUs (node of 8): huge gradients and tiny activations ->
    # the most tensor parallelism (less all-reduce); huge activations and tiny
    # gradients -> none
    big_p = _workload(_layers(4, t=1e-3, p=4e9, a=1e3, x=1.0), 64, [8], [2], mem=1e13)
    g = px.grid(big_p, 0, 0, 8, 1.0, 1, 2, F_REF)
    assert g["ok"] and list(g["Dn"]) == [8] and list(g["tp"]) == [8]
    big_x = _workload(_layers(4, t=1e-3, p=1.0, a=1e3, x=1e9), 64, [8], [2], mem=1e13)
    g = px.grid(big_x, 0, 0, 8, 1.0, 1, 2, F_REF)
    assert g["ok"] and list(g["tp"]) == [1]


def test_memory_moves_the_proxy_to_more_stages():
    # 8 layers of 20 GB parameters: one stage needs 640 GB / tp of optimizer
    # state on 8 GPUs of 100 GB (tp <= 4 in a node of 4) -> no single-stage
    # plan fits; the cell's proxy uses several stages
    w = _workload(_layers(8, t=1e-3, p=2e10, a=1e3), 64, [8], [1, 2, 4], mem=1e11, gpn=4)
    for B in (1, 2, 4):
        assert not px.grid(w, 0, 0, 8, 1.0, 1, B, F_REF)["ok"]
    r = px.cells(w, [0])
    assert np.isfinite(r["T"][0]) and r["s"][0] >= 2


def test_grid_proxy_is_the_least_bias_over_every_grouping():
    # enumerate the groupings independently (itertools) and normalise each:
    # the grid's proxy has the least bias among those that fit
    rng = np.random.default_rng(7)
    L = 7
    w = _workload(dict(t=list(rng.uniform(1e-3, 9e-3, L)), p=list(rng.uniform(1e7, 1e8, L)),
                       a=list(rng.uniform(1e4, 1e5, L)), x=list(rng.uniform(1e4, 1e5, L)),
                       a2a=[0.0] * L), 64, [16], [2], mem=1e13)
    _, d = px.loads(w, 0, 0, 16, F_REF)
    for s in range(1, 8):
        best = math.inf
        for cuts in itertools.combinations(range(1, L), s - 1):
            b = [0, *cuts, L]
            D = []
            for j in range(s):
                acc = 0.0
                for i in range(b[j], b[j + 1]):
                    acc += float(d[i])
                D.append(acc)
            b2, _ = px.normalize(D, 16)
            if b2 is not None:
                best = min(best, b2)
        g = px.grid(w, 0, 0, 16, 1.0, s, 2, F_REF)
        if math.isinf(best):
            assert not g["ok"]
        else:
            assert g["ok"] and g["b2"] == best


def test_cell_takes_the_best_grid_with_the_tie_rule():
    w = wl.make("small").subset_jobs([3, 17])
    kap = float(w.kappa[0][0])
    for j in range(2):
        for ci in (3, 5, 6):
            n = int(w.counts[ci])
            cell = (j * w.n_types + 0) * w.n_counts + ci
            r = px.cells(w, [cell])
            grids = {}
            for s in range(1, min(16, w.layers(j), n) + 1):
                for B in w.m_values:
                    g = px.grid(w, j, 0, n, float(w.kappa[0][ci]), s, int(B), F_REF)
                    if g["ok"]:
                        grids[(s, int(B))] = g["T"]
            if not grids:
                assert not np.isfinite(r["T"][0])
                continue
            tmin = min(grids.values())
            pick = min(k for k, v in grids.items() if v <= tmin * (1 + w.tie_eps))
            assert (int(r["s"][0]), int(r["B"][0])) == pick
            assert r["T"][0] == grids[pick]
    del kap


def test_uniform_proxies_price_as_the_uniform_oracle():
    # a proxy whose stages are alike is a plan of the uniform space: its price
    # equals the uniform oracle's price of the same (dp, tp, pp, m) with the
    # proxy's cuts (operator boundaries mapped to layers)
    w = wl.make("small")
    ids = np.arange(0, w.n_cells, 11)
    r = px.cells(w, ids)
    checked = 0
    for q, cell in enumerate(ids):
        s = int(r["s"][q])
        if s == 0:
            continue
        Dn, tp = r["Dn"][q][:s], r["tp"][q][:s]
        if len(set(Dn)) != 1 or len(set(tp)) != 1:
            continue
        ci = int(cell % w.n_counts)
        g = int((cell // w.n_counts) % w.n_types)
        j = int(cell // (w.n_counts * w.n_types))
        L = w.layers(j)
        O = min(L, 16)
        cuts = [(int(b) * L) // O for b in r["bounds"][q][1:s]]
        n = int(w.counts[ci])
        ref = uo.eval_plan(w, j, g, n, float(w.kappa[0][g * w.n_counts + ci]), int(Dn[0] // tp[0]),
                           int(tp[0]), s, int(r["B"][q]), cuts=cuts)
        assert ref["feasible"]
        assert r["T"][q] == pytest.approx(ref["T"], rel=1e-12)
        checked += 1
    assert checked > 10


# ---------------------------------------------------------------- hand-derived tie-breaks

def test_bias_tie_takes_the_larger_multiset():
    # shares (3, 1.5, 1.5) on 6 GPUs: {4, 1, 1} and {2, 2, 2} both have squared
    # bias 1 + 0.25 + 0.25 = 1.5; the lexicographically larger sorted multiset wins
    b2, m = px.normalize([3.0, 1.5, 1.5], 6)
    assert b2 == 1.5 and list(m) == [4, 1, 1]


def _three_ops(a2a):
    # three layers (= operators) of compute time 1, 2, 1: shares 1, 2, 1 of 4
    # GPUs; no memory traffic, no weights; huge TP volume so tp 1 is chosen
    return _workload(dict(t=[1.0, 2.0, 1.0], p=[0.0] * 3, a=[0.0] * 3, x=[1e9] * 3, a2a=a2a), 8, [4], [2],
                     bwi=1e9, bwe=1e9, gpn=2, mem=1e15, hbm=1e30)


def test_communication_load_breaks_a_bias_tie_with_its_pipeline_term():
    """Groupings {0}{1,2} and {0,1}{2} both get 2 + 2 GPUs (shares (1, 3) and
    (3, 1): squared bias 2 each).  With B = 2 each stage is dp 2 x tp 1 with
    b = 8 / (2 x 2) = 2 samples per microbatch and all-to-all volumes
    (0, 1e9, 2e9) at 1e9 B/s: C = 2 x (sum a2a) / 1e9.
      {0}{1,2}:  C = (0, 6): l_comm = (2-1) x 6 + 6 = 12
      {0,1}{2}:  C = (2, 4): l_comm = (2-1) x 4 + 6 = 10
    The sums tie; the (B-1) max C term picks the second grouping."""
    g = px.grid(_three_ops([0.0, 1e9, 2e9]), 0, 0, 4, 1.0, 2, 2, F_REF)
    assert g["ok"] and g["b2"] == 2.0
    assert list(g["bounds"]) == [0, 2, 3] and list(g["Dn"]) == [2, 2] and list(g["tp"]) == [1, 1]
    assert g["lcomm"] == pytest.approx(10.0, rel=1e-12)


def test_full_tie_keeps_the_first_grouping():
    # no communication at all: both groupings have bias 2 and l_comm 0; the
    # lexicographically smallest cut vector ({0}{1,2}) is the proxy
    g = px.grid(_three_ops([0.0, 0.0, 0.0]), 0, 0, 4, 1.0, 2, 2, F_REF)
    assert g["ok"] and list(g["bounds"]) == [0, 1, 3] and g["lcomm"] == 0.0


def test_equal_intra_stage_costs_take_the_smaller_tp():
    # one stage of 2 GPUs (node of 2) with no communication of any kind: tp 1
    # and tp 2 cost 0 each; the smaller tensor degree is kept
    w = _workload(dict(t=[1.0, 1.0], p=[0.0, 0.0], a=[0.0, 0.0], x=[0.0, 0.0], a2a=[0.0, 0.0]), 2, [2], [1],
                  bwi=1e9, bwe=1e9, gpn=2, mem=1e15, hbm=1e30)
    g = px.grid(w, 0, 0, 2, 1.0, 1, 1, F_REF)
    assert g["ok"] and list(g["Dn"]) == [2] and list(g["tp"]) == [1]


def test_p2p_between_unequal_stages_carries_the_smaller_replica_count():
    """Two layers of time 1, batch 4, B = 2; stage 0 on 2 GPUs (dp 2, b = 1),
    stage 1 on 1 GPU (b = 2); x = (0.25, 0) at 1 B/s inside a node of 4.
    W0 = 1 x 1/4, W1 = 2 x 1/4; the boundary carries the samples of the smaller
    dp: 2 x (4 / (1 x 2)) x 0.25 = 1.  T = (0.25 + 1) + 0.5 + (2-1) x 0.5 = 2.25."""
    w = _workload(dict(t=[1.0, 1.0], p=[0.0, 0.0], a=[0.0, 0.0], x=[0.25, 0.0], a2a=[0.0, 0.0]), 4, [3], [2],
                  bwi=1.0, bwe=1.0, gpn=4, mem=1e15, hbm=1e30)
    T, feas, _ = px.price(w, 0, 0, 3, 1.0, [0, 1, 2], [2, 1], [1, 1], 2, F_REF)
    assert feas and T == 2.25
