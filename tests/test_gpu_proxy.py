"""Parity of the HIP proxy-plan planner (arena_proxy_estimate) with its CPU
oracle, through the C ABI.

Every decision (bias, feasibility, communication load, grid choice) is taken
in fp64 in the same operation order on both sides, so the plan of every cell
-- stage count, microbatch count, stage boundaries, GPUs and tensor degree of
each stage -- must be identical, and the iteration time equal up to its f32
rounding (1e-6 relative is asserted)."""
import numpy as np
import pytest

from oracle import proxy as px
from paper_2403_16125_amd import workloads as wl

pytestmark = pytest.mark.gpu

F_REF = wl.F_REF
REL_T = 1e-6


def _gpu(w, ids, kappa_round=0, n_ops=16):
    from paper_2403_16125_amd import arena
    est = arena.Estimator(w, device=0)
    try:
        est.set_round(kappa_round)
        est.proxy_estimate(f_ref=F_REF, n_ops=n_ops)
        return est.proxy_results(ids)
    finally:
        est.close()


def _bounds_mask(bounds, s):
    m = 0
    for b in bounds[1:s]:
        m |= 1 << (int(b) - 1)
    return m


def _compare(w, ids, kappa_round=0, n_ops=16):
    print(f"proxy parity: {w.name}, {len(ids)} cells, round {kappa_round}, n_ops {n_ops}", flush=True)
    got = _gpu(w, ids, kappa_round, n_ops)
    want = px.cells(w, ids, kappa_round=kappa_round, f_ref=F_REF, n_ops=n_ops)
    bad = []
    for q in range(len(ids)):
        T = float(want["T"][q])
        if not np.isfinite(T):
            if got["feasible"][q] or np.isfinite(got["t_iter"][q]) or got["thr"][q] != 0 or got["words"][q].any():
                bad.append((int(ids[q]), "infeasible cell with outputs"))
            continue
        s = int(want["s"][q])
        same = (got["feasible"][q] and int(got["s"][q]) == s and int(got["B"][q]) == int(want["B"][q])
                and int(got["starts"][q]) == _bounds_mask(want["bounds"][q], s)
                and list(got["Dn"][q][:s]) == list(want["Dn"][q][:s])
                and list(got["tp"][q][:s]) == list(want["tp"][q][:s]))
        if not same:
            bad.append((int(ids[q]), "plan differs", s, int(got["s"][q])))
            continue
        if abs(float(got["t_iter"][q]) - T) > REL_T * T or \
                abs(float(got["thr"][q]) - float(want["thr"][q])) > REL_T * float(want["thr"][q]):
            bad.append((int(ids[q]), "T differs", T, float(got["t_iter"][q])))
    assert not bad, f"{len(bad)} of {len(ids)} cells differ: {bad[:5]}"
    return got, want


def test_tiny_every_cell():
    w = wl.make("tiny")
    _compare(w, np.arange(w.n_cells))


def test_small_every_cell():
    w = wl.make("small")
    got, want = _compare(w, np.arange(w.n_cells))
    # the sample exercises several stage counts and uneven stage GPU counts
    s = want["s"][np.isfinite(want["T"])]
    assert len(np.unique(s)) >= 8
    uneven = [q for q in range(len(s)) if len(set(want["Dn"][q][:want["s"][q]])) > 1]
    assert len(uneven) > 50


@pytest.mark.parametrize("name,step", [("trace", 977), ("moe", 4099)])
def test_sampled_cells(name, step):
    w = wl.make(name)
    _compare(w, np.arange(0, w.n_cells, step))


def test_other_operator_counts_and_rounds():
    w = wl.make("small")
    ids = np.arange(0, w.n_cells, 5)
    _compare(w, ids, n_ops=4)
    _compare(w, ids, n_ops=1)
    w = wl.make("trace").subset_jobs(range(0, 1024, 64))
    _compare(w, np.arange(w.n_cells), kappa_round=0)


def test_edge_jobs():
    # one layer, zero-cost layers, a job with no load at all, a job too large
    # for any grid, counts that are no power of two, a node of 3 GPUs
    rng = np.random.default_rng(5)
    jobs = [
        dict(batch=32, t=[2e-3], p=[1e8], a=[1e6], x=[1e5], a2a=[0.0]),
        dict(batch=64, t=[0.0, 1e-3, 0.0, 2e-3, 0.0], p=[0.0, 1e8, 0.0, 1e8, 0.0], a=[0.0, 1e6, 0.0, 1e6, 0.0],
             x=[1e5] * 5, a2a=[0.0] * 5),
        dict(batch=16, t=[0.0] * 6, p=[0.0] * 6, a=[0.0] * 6, x=[0.0] * 6, a2a=[0.0] * 6),
        dict(batch=128, t=list(rng.uniform(1e-3, 5e-3, 20)), p=[5e11] * 20, a=[1e9] * 20,
             x=[1e6] * 20, a2a=[0.0] * 20),
        dict(batch=96, t=list(rng.uniform(1e-3, 5e-3, 40)), p=list(rng.uniform(1e8, 1e9, 40)),
             a=list(rng.uniform(1e5, 1e7, 40)), x=list(rng.uniform(1e4, 1e6, 40)),
             a2a=list(np.where(np.arange(40) % 2 == 1, 3e5, 0.0))),
    ]
    types = [dict(speed=1.0, mem=80e9, bw_intra=300e9, bw_inter=25e9, gpus_per_node=8),
             dict(speed=0.4, mem=24e9, bw_intra=64e9, bw_inter=12.5e9, gpus_per_node=3)]
    w = wl.from_lists(jobs, types, [1, 2, 3, 6, 12, 24, 40], [1, 2, 3, 4, 8, 16], kappa=1.2)
    got, want = _compare(w, np.arange(w.n_cells))
    per_job = w.n_types * w.n_counts
    assert not np.isfinite(want["T"][2 * per_job:3 * per_job]).any()    # no load: no proxy
    assert not np.isfinite(want["T"][3 * per_job:4 * per_job]).any()    # fits nowhere


def test_full_round_jobs_every_grid():
    # jobs of the full scheduling round (trace-like and MoE mixed, 8 types x
    # 131 counts up to 1024 GPUs, contention redrawn per round): every grid of
    # 24 jobs runs on the GPU, a sample of cells is checked
    w = wl.make("full").subset_jobs(range(0, 16384, 683))
    ids = np.arange(0, w.n_cells, 97)
    _compare(w, ids, kappa_round=3)


def _hand(layers, batch, counts, m_values, gpn, bw):
    ty = dict(speed=1.0, mem=1e15, bw_intra=bw, bw_inter=bw, gpus_per_node=gpn)
    w = wl.from_lists([dict(batch=batch, **layers)], [ty], counts, m_values, kappa=1.0)
    w.hbm = np.asarray([1e30], np.float32)
    return w


def test_hand_tie_workloads():
    """The hand-derived tie cases of the oracle's pins (a bias tie decided by the
    pipeline term of the communication load, a full tie kept by the first
    grouping, equal intra-stage costs keeping the smaller tp, p2p between
    unequal stages) as whole cells over several GPU counts."""
    three = lambda a2a: dict(t=[1.0, 2.0, 1.0], p=[0.0] * 3, a=[0.0] * 3, x=[1e9] * 3, a2a=a2a)
    cases = [
        _hand(three([0.0, 1e9, 2e9]), 8, [2, 3, 4], [1, 2], 2, 1e9),
        _hand(three([0.0, 0.0, 0.0]), 8, [2, 3, 4], [1, 2], 2, 1e9),
        _hand(dict(t=[1.0, 1.0], p=[0.0, 0.0], a=[0.0, 0.0], x=[0.0, 0.0], a2a=[0.0, 0.0]), 2, [1, 2], [1], 2, 1e9),
        _hand(dict(t=[1.0, 1.0], p=[0.0, 0.0], a=[0.0, 0.0], x=[0.25, 0.0], a2a=[0.0, 0.0]), 4, [2, 3, 4], [1, 2],
              4, 1.0),
    ]
    for w in cases:
        _compare(w, np.arange(w.n_cells))
