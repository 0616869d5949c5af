"""Pins of the oracle's interpolated communication latency (CPU only).

Communication latency is profiled per primitive at sampled volumes and
interpolated by volume online (Sec. 3.4).  Here each GPU type has one table
per link (inside a node, across nodes) and every communication term takes its
latency from the table of its link; a plan's per-microbatch layer costs then
depend on its microbatch size, so each plan gets its own balanced partition.
Fixed outside the oracle's code:
  * the interpolation on a hand table (inside, at and beyond the samples, a
    start-up offset, nothing moved);
  * tables linear through the origin reproduce the volume / bandwidth model
    (the same cells, plans and cuts);
  * hand-derived plan prices and the cell's choice;
  * slower tables never make a cell faster;
  * an enumeration of every plan and cut vector of small cells.
"""
import itertools
import math

import numpy as np
import pytest

from paper_2403_16125_amd import workloads as wl

INF = math.inf


def test_interpolation_on_a_hand_table(oracle):
    vol, lat = [0.0, 10.0, 20.0], [0.0, 1.0, 5.0]
    assert oracle.tab_latency(vol, lat, 5.0) == 0.5      # inside the first segment
    assert oracle.tab_latency(vol, lat, 10.0) == 1.0     # at a sample
    assert oracle.tab_latency(vol, lat, 15.0) == 3.0     # second segment
    assert oracle.tab_latency(vol, lat, 30.0) == 9.0     # last segment extended
    assert oracle.tab_latency(vol, lat, 0.0) == 0.0      # nothing moves
    off = ([0.0, 10.0], [0.5, 1.5])                      # start-up cost 0.5
    assert oracle.tab_latency(*off, 2.0) == pytest.approx(0.7, rel=1e-15)
    assert oracle.tab_latency(*off, 0.0) == 0.0


@pytest.mark.parametrize("name,step", [("small", 1), ("trace", 211), ("moe", 397)])
def test_linear_tables_reproduce_the_bandwidth_model(oracle, name, step):
    w = wl.make(name)
    ids = np.arange(0, w.n_cells, step)
    r0 = oracle.cells(w, ids)
    r1 = oracle.cells_tab(w, ids, wl.linear_tables(w, K=3))
    for k in ("dp", "tp", "pp", "m"):
        assert np.array_equal(r0[k], r1[k]), k
    assert np.array_equal(r0["cuts"], r1["cuts"])
    fin = np.isfinite(r0["T"])
    assert np.array_equal(fin, np.isfinite(r1["T"]))
    assert np.allclose(r1["T"][fin], r0["T"][fin], rtol=1e-12, atol=0)


def _hand():
    # two layers of time 1 (batch 2), boundary activations 5e8 B, weights
    # 2.5e8 B each, no activations stored, 2 GPUs on one node of 2; both links
    # share the table (0, 0.25 s), (5e8 B, 0.65 s), (1e9 B, 1.25 s)
    job = dict(t=[1.0, 1.0], p=[2.5e8, 2.5e8], a=[0.0, 0.0], x=[5e8, 5e8], a2a=[0.0, 0.0], batch=2)
    ty = dict(speed=1.0, mem=1e15, bw_intra=1e9, bw_inter=1e9, gpus_per_node=2)
    w = wl.from_lists([job], [ty], [2], [1, 2], kappa=1.0)
    v = np.array([0.0, 5e8, 1e9])
    l = np.array([0.25, 0.65, 1.25])
    vol = np.broadcast_to(v, (1, 2, 3)).copy()
    lat = np.broadcast_to(l, (1, 2, 3)).copy()
    return w, (vol, lat)


def test_hand_plan_prices(oracle):
    """(dp, tp, pp, m) = (1, 2, 1, 1): b = 2; each layer computes 2 x 1/(2 x 2) =
      0.5 and runs 4 all-reduces of 2 (1/2) 2 x 5e8 = 1e9 B: 4 x 1.25; T = 2 x 5.5 = 11.
    (1, 1, 2, 2): b = 1; stages of 0.5 each, the boundary moves 5e8 B twice:
      2 x 0.65 = 1.3; T = (0.5 + 1.3) + 0.5 + (2 - 1) x 0.5 = 2.8.
    (2, 1, 1, 1): b = 1; 0.5 + 0.5 = 1 of compute, gradient all-reduce of
      2 (1/2) 5e8 = 5e8 B: 0.65; T = 1.65 (the cell's best)."""
    w, tabs = _hand()
    assert oracle.eval_plan_tab(w, 0, 0, 2, 1.0, 1, 2, 1, 1, tabs)["T"] == 11.0
    e = oracle.eval_plan_tab(w, 0, 0, 2, 1.0, 1, 1, 2, 2, tabs)
    assert e["T"] == pytest.approx(2.8, rel=1e-15) and e["cuts"] == [1]
    assert oracle.eval_plan_tab(w, 0, 0, 2, 1.0, 2, 1, 1, 1, tabs)["T"] == pytest.approx(1.65, rel=1e-15)
    r = oracle.cells_tab(w, [0], tabs)
    assert (r["dp"][0], r["tp"][0], r["pp"][0], r["m"][0]) == (2, 1, 1, 1)
    # five plans: the three above, (1, 2, 1, 2) and (1, 1, 2, 1)
    assert r["T"][0] == pytest.approx(1.65, rel=1e-15) and r["nplans"][0] == 5


def test_slower_tables_never_make_a_cell_faster(oracle):
    w = wl.make("small")
    ids = np.arange(w.n_cells)
    vol, lat = wl.comm_tables(w)
    r1 = oracle.cells_tab(w, ids, (vol, lat))
    r2 = oracle.cells_tab(w, ids, (vol, lat * 1.5))
    fin = np.isfinite(r1["T"])
    assert np.array_equal(fin, np.isfinite(r2["T"]))
    assert np.all(r2["T"][fin] >= r1["T"][fin])
    assert np.sum(r2["T"][fin] > r1["T"][fin]) > 0.5 * fin.sum()


def _enumerate_cell(o, w, ci, tabs):
    n = int(w.counts[ci])
    L = int(w.layer_offset[1] - w.layer_offset[0])
    gpn, bg = int(w.gpus_per_node[0]), int(w.batch[0])
    kap = float(w.kappa[0][ci])
    cands = []
    for tp in range(1, n + 1):
        if n % tp or tp > gpn or gpn % tp:
            continue
        for pp in range(1, n // tp + 1):
            if (n // tp) % pp or pp > L:
                continue
            dp = n // (tp * pp)
            for m in (int(v) for v in w.m_values):
                if bg % (dp * m):
                    continue
                best = None
                for cuts in itertools.combinations(range(1, L), pp - 1):
                    e = o.eval_plan_tab(w, 0, 0, n, kap, dp, tp, pp, m, tabs, cuts=list(cuts))
                    if best is None or e["w_max"] < best[0]:
                        best = (e["w_max"], e, list(cuts))
                e = best[1]
                if e["feasible"]:
                    cands.append((e["T"], pp, tp, m, dp, best[2]))
    if not cands:
        return None
    tmin = min(c[0] for c in cands)
    return min((c for c in cands if c[0] <= tmin * (1 + float(w.tie_eps))), key=lambda c: (c[1], c[2], c[3]))


def test_small_cells_against_enumeration(oracle):
    rng = np.random.default_rng(8)
    checked = 0
    for trial in range(30):
        L = int(rng.integers(2, 8))
        job = dict(t=list(rng.lognormal(0, 0.7, L)), p=list(rng.lognormal(19, 1.0, L)),
                   a=list(rng.lognormal(16, 1.0, L)), x=list(rng.lognormal(17, 1.0, L)),
                   a2a=list(rng.lognormal(16, 1.0, L) * (rng.random(L) < 0.5)), batch=int(rng.choice([4, 8, 16])))
        tot = 4 * sum(job["p"]) + job["batch"] * sum(job["a"])
        ty = dict(speed=1.0, mem=float(tot * rng.uniform(0.2, 1.5)), bw_intra=2e10, bw_inter=2.5e9,
                  gpus_per_node=int(rng.choice([1, 2, 4])))
        counts = [1, 2, 3, 4, 6, 8]
        w = wl.from_lists([job], [ty], counts, [1, 2, 4, 8], kappa=float(rng.uniform(1.0, 2.0)))
        tabs = wl.comm_tables(w)
        r = oracle.cells_tab(w, range(len(counts)), tabs)
        for ci in range(len(counts)):
            want = _enumerate_cell(oracle, w, ci, tabs)
            checked += 1
            if want is None:
                assert r["T"][ci] == INF and r["pp"][ci] == 0
                continue
            T, pp, tp, m, dp, cuts = want
            assert (r["dp"][ci], r["tp"][ci], r["pp"][ci], r["m"][ci]) == (dp, tp, pp, m)
            assert r["T"][ci] == T and list(r["cuts"][ci][:pp - 1]) == cuts
    assert checked == 180
