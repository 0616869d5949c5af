"""Pins of the scheduler oracle (CPU): hand-derived steps of Algorithm 1 under
the throughput objective (Eq. 5), and invariants on random cluster states."""
import numpy as np
import pytest

from oracle import scheduler_oracle as so
from paper_2403_16125_amd import sched_states as ss


def _thr(rows):
    """rows: {job: [[thr per count] per type]} -> f32 [J, T, NC]"""
    J = max(rows) + 1
    T = len(next(iter(rows.values())))
    NC = len(next(iter(rows.values()))[0])
    a = np.zeros((J, T, NC), np.float32)
    for j, r in rows.items():
        a[j] = np.asarray(r, np.float32)
    return a


def test_launch_takes_the_fastest_grid_that_fits():
    thr = _thr({0: [[10, 18, 30], [12, 20, 25]]})
    r = so.schedule(thr, [1, 2, 4], [4, 4], [-1], [0], [0], [0], 4)
    assert r["launched"] == [1] and (r["alloc_type"][0], r["alloc_count"][0]) == (0, 2)
    # only 2 GPUs of type 0 free: type 1 with 4 GPUs (25) beats type 0 with 2 (18)
    r = so.schedule(thr, [1, 2, 4], [2, 4], [-1], [0], [0], [0], 4)
    assert (r["alloc_type"][0], r["alloc_count"][0]) == (1, 2)


def test_launch_ties_go_to_fewer_gpus_then_lower_type():
    thr = _thr({0: [[10, 20, 20], [5, 20, 20]]})
    r = so.schedule(thr, [1, 2, 4], [4, 4], [-1], [0], [0], [0], 4)
    assert (r["alloc_type"][0], r["alloc_count"][0]) == (0, 1)


def _scale_down_case():
    # job 0 queued (needs 2 GPUs); jobs 1 and 2 each run on 2 of the 4 GPUs.
    # Scaling job 1 from 2 to 1 GPU costs 19 - 10 = 9 per GPU, job 2 costs 20 - 3 = 17.
    thr = _thr({0: [[0, 50, 80]], 1: [[10, 19, 0]], 2: [[3, 20, 0]]})
    return thr, [1, 2, 4], [4], [-1, 0, 0], [0, 1, 1], [0], [0]


def test_scale_down_cheapest_first_until_the_job_fits():
    thr, counts, cap, at, ac, q, p = _scale_down_case()
    r = so.schedule(thr, counts, cap, at, ac, q, p, 4)
    # job 1 goes to 1 GPU (cost 9), one GPU is not enough, job 1 has no smaller
    # count left, so job 2 goes to 1 GPU (cost 17); job 0 then runs on 2 GPUs
    assert r["launched"] == [1]
    assert r["alloc_count"] == [1, 0, 0] and r["alloc_type"] == [0, 0, 0]
    assert r["moves"] == [2, 1, 0]
    # searches: launch (fails), scale-down, launch (fails), scale-down, launch,
    # then one scale-up search that finds no free GPU
    assert r["decisions"] == 6


def test_scale_downs_are_undone_when_the_depth_runs_out():
    thr, counts, cap, at, ac, q, p = _scale_down_case()
    r = so.schedule(thr, counts, cap, at, ac, q, p, 1)
    assert r["launched"] == [0]
    assert r["alloc_count"] == [0, 1, 1] and r["alloc_type"] == [-1, 0, 0]
    assert r["moves"] == [0, 0, 0]
    assert r["decisions"] == 4      # launch, scale-down, launch, (undo), scale-up search


def test_scale_down_only_on_types_the_queued_job_can_use():
    # job 0 only runs on type 1; the cheap scale-down sits on type 0
    thr = _thr({0: [[0, 0], [0, 40]], 1: [[10, 11], [0, 0]], 2: [[0, 0], [5, 30]]})
    r = so.schedule(thr, [1, 2], [2, 2], [-1, 0, 1], [0, 1, 1], [0], [0], 4)
    # stepping job 2 down frees one GPU of type 1, not enough for job 0: undone;
    # job 1 (type 0, useless to job 0) is never touched
    assert r["launched"] == [0]
    assert r["alloc_count"] == [0, 1, 1]
    # with 3 GPUs of type 1 the one freed GPU is enough: one scale-down (job 2),
    # one launch, no scale-up, and job 1 never moved (stepping it down and back
    # up again would end in the same allocation, so the moves are checked too)
    r = so.schedule(thr, [1, 2], [2, 3], [-1, 0, 1], [0, 1, 1], [0], [0], 4)
    assert r["launched"] == [1] and r["alloc_count"][2] == 0 and r["alloc_count"][1] == 1
    assert r["moves"] == [1, 1, 0] and r["decisions"] == 4


def test_scale_down_cost_is_per_freed_gpu():
    # one type of 6 GPUs, counts 1, 2, 4; job 1 runs on 4 (4 -> 2 loses 30 - 20
    # = 10 for 2 GPUs: 5 per GPU), job 2 on 2 (2 -> 1 loses 10 - 2 = 8 for 1 GPU:
    # 8 per GPU); queued job 0 needs 2.  Per freed GPU, job 1 is cheaper: one
    # scale-down, job 0 launches on 2, nothing left to scale up
    thr = _thr({0: [[0, 50, 80]], 1: [[5, 20, 30]], 2: [[2, 10, 0]]})
    r = so.schedule(thr, [1, 2, 4], [6], [-1, 0, 0], [0, 2, 1], [0], [0], 4)
    assert r["launched"] == [1]
    assert r["alloc_count"] == [1, 1, 1] and r["moves"] == [1, 1, 0] and r["decisions"] == 4


def test_first_failed_launch_sets_the_allowance():
    # queue: job 0 (class 1) needs 4 GPUs of the 2 there are and fails, which
    # allows class <= 1 from then on; job 1 (class 1) fits on one GPU
    thr = _thr({0: [[0, 0, 50]], 1: [[10, 0, 0]]})
    r = so.schedule(thr, [1, 2, 4], [2], [-1, -1], [0, 0], [0, 1], [1, 1], 4)
    assert r["launched"] == [0, 1] and r["alloc_type"] == [-1, 0] and r["alloc_count"] == [0, 0]


def test_deadline_met_exactly_is_open():
    # batch 4 x 10 iterations = 40 samples; at 20 samples/s (2 GPUs) the job
    # finishes in exactly its 2 s deadline: open; at 10 samples/s (1 GPU) not
    thr = _thr({0: [[10, 20]]})
    r = so.schedule(thr, [1, 2], [2], [-1], [0], [0], [0], 4, batch=[4], iters=[10.0], deadline=[2.0])
    assert r["launched"] == [1] and r["alloc_count"] == [1]
    r = so.schedule(thr, [1, 2], [2], [-1], [0], [0], [0], 4, batch=[4], iters=[10.0], deadline=[1.999])
    assert r["launched"] == [0]


def test_priority_rule_stops_after_a_failed_class():
    # one type, 2 GPUs; a (class 0) takes both; b (class 0) fails and sets
    # lam' = 0; c (class 1) fails -> stop; d (class 1, would fit on 1 GPU of a
    # free cluster) is never visited
    thr = _thr({0: [[0, 9]], 1: [[5, 8]], 2: [[0, 7]], 3: [[4, 0]]})
    r = so.schedule(thr, [1, 2], [2], [-1] * 4, [0] * 4, [0, 1, 2, 3], [0, 0, 1, 1], 4)
    assert r["launched"] == [1, 0, 0, 0]
    # same class: a failed job does not stop the visit
    thr2 = _thr({0: [[0, 9]], 1: [[0, 8]], 2: [[0, 0]], 3: [[4, 0]]})
    r = so.schedule(thr2, [1, 2], [3], [-1] * 4, [0] * 4, [0, 1, 2, 3], [0, 0, 0, 0], 4)
    assert r["launched"] == [1, 0, 0, 1]


def test_scale_up_best_gain_per_gpu_first():
    thr = _thr({0: [[5, 9, 16, 20]], 1: [[4, 10, 19, 30]]})
    r = so.schedule(thr, [1, 2, 4, 8], [8], [0, 0], [1, 1], [], [], 8)
    # free 4: job 1 to 4 GPUs (gain 4.5/GPU) beats job 0 (3.5/GPU); then job 0 to 4
    assert r["alloc_count"] == [2, 2] and r["moves"] == [0, 0, 2] and r["free"] == [0]
    r = so.schedule(thr, [1, 2, 4, 8], [8], [0, 0], [1, 1], [], [], 1)
    assert r["alloc_count"] == [1, 2] and r["moves"] == [0, 0, 1]


def test_scale_up_takes_the_best_step_not_the_next():
    # from 1 GPU: to 2 gains 1/GPU, to 4 gains (40 - 10) / 3 = 10/GPU
    thr = _thr({0: [[10, 11, 40]]})
    r = so.schedule(thr, [1, 2, 4], [4], [0], [0], [], [], 4)
    assert r["alloc_count"] == [2]


def test_rejects_bad_states():
    thr = _thr({0: [[1, 2]], 1: [[1, 2]]})
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [2], [0, 0], [1, 1], [], [], 1)     # 4 GPUs busy of 2
    with pytest.raises(ValueError):
        so.schedule(thr, [2, 1], [4], [-1, -1], [0, 0], [], [], 1)   # counts not ascending
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [4], [0, -1], [0, 0], [0], [0], 1)   # queued job already running
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [4], [-1, -1], [0, 0], [1, 1], [0, 0], 1)   # listed twice
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [4], [-1, -1], [0, 0], [1], [-1], 1)        # negative class


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_invariants_on_random_states(seed):
    counts = [1, 2, 4, 8, 16, 32]
    thr = ss.synthetic_thr(seed, 60, 3, counts)
    st = ss.random_state(seed, thr, counts, [40, 24, 16], running_frac=0.5, queued_frac=0.3, depth=4)
    r = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue,
                    st.priority, st.depth)
    used = np.zeros(3, np.int64)
    for j in range(st.n_jobs):
        g = r["alloc_type"][j]
        if g >= 0:
            used[g] += counts[r["alloc_count"][j]]
            assert st.thr[j, g, r["alloc_count"][j]] > 0 or st.alloc_type[j] == g
            if st.alloc_type[j] >= 0:
                assert g == st.alloc_type[j]        # running jobs keep their type
    assert (used <= st.capacity).all()
    assert list(used + np.asarray(r["free"])) == list(st.capacity)
    assert r["moves"][2] <= st.depth
    for q, j in enumerate(st.queue):
        assert (r["alloc_type"][j] >= 0) == bool(r["launched"][q])


def test_deadline_gates_the_launch():
    # B N = 300: 1, 2, 4 GPUs finish in 30, 16.7, 10 s; a 12 s deadline opens only 4 GPUs
    thr = _thr({0: [[10, 18, 30]]})
    kw = dict(batch=[10], iters=[30.0], deadline=[12.0])
    r = so.schedule(thr, [1, 2, 4], [4], [-1], [0], [0], [0], 4, **kw)
    assert r["launched"] == [1] and r["alloc_count"] == [2]
    r = so.schedule(thr, [1, 2, 4], [2], [-1], [0], [0], [0], 4, **kw)     # 2 GPUs fit, but too slow
    assert r["launched"] == [0] and r["alloc_type"] == [-1]
    r = so.schedule(thr, [1, 2, 4], [2], [-1], [0], [0], [0], 4)           # no deadline: launches on 2
    assert r["launched"] == [1] and r["alloc_count"] == [1]


def test_deadline_protects_a_scale_down():
    # the scale-down case with job 1 (the cheapest to shrink) unable to finish on 1 GPU in
    # time: only job 2 may shrink, which frees one GPU, not enough, so job 0 waits and the
    # move is undone; with a roomier deadline for job 1 the original two scale-downs return
    thr, counts, cap, at, ac, q, p = _scale_down_case()
    base = dict(batch=[1, 1, 1], iters=[1.0, 100.0, 1.0])
    r = so.schedule(thr, counts, cap, at, ac, q, p, 4, deadline=[1e9, 6.0, 1e9], **base)
    # job 1 on 1 GPU needs 100 / 10 = 10 s > 6 s: not open; job 2 to 1 GPU frees one GPU only
    assert r["launched"] == [0] and r["alloc_count"] == [0, 1, 1] and r["moves"] == [0, 0, 0]
    r = so.schedule(thr, counts, cap, at, ac, q, p, 4, deadline=[1e9, 20.0, 1e9], **base)
    assert r["launched"] == [1] and r["alloc_count"] == [1, 0, 0] and r["moves"] == [2, 1, 0]


def test_deadline_steers_a_scale_up():
    # 1 -> 2 and 1 -> 4 GPUs gain 1 sample/s per GPU alike (tie: the smaller count); a
    # deadline that only 4 GPUs meet makes 4 the move
    thr = _thr({0: [[1, 2, 4]]})
    r = so.schedule(thr, [1, 2, 4], [4], [0], [0], [], [], 1)
    assert r["alloc_count"] == [1]
    r = so.schedule(thr, [1, 2, 4], [4], [0], [0], [], [], 1, batch=[1], iters=[10.0], deadline=[3.0])
    assert r["alloc_count"] == [2]


def test_deadline_values_checked_and_infinite_is_none():
    thr = _thr({0: [[1, 2]], 1: [[1, 2]]})
    for bad in (dict(batch=[0, 1], iters=[1.0, 1.0], deadline=[1.0, 1.0]),
                dict(batch=[1, 1], iters=[-1.0, 1.0], deadline=[1.0, 1.0]),
                dict(batch=[1, 1], iters=[1.0, 1.0], deadline=[0.0, 1.0]),
                dict(batch=[1, 1], iters=[1.0, 1.0], deadline=[float("nan"), 1.0]),
                dict(batch=[1, 1], iters=[1.0, 1.0])):
        with pytest.raises(ValueError):
            so.schedule(thr, [1, 2], [4], [-1, -1], [0, 0], [0], [0], 1, **bad)
    counts = [1, 2, 4, 8, 16, 32]
    thr = ss.synthetic_thr(9, 80, 3, counts)
    st = ss.random_state(9, thr, counts, [40, 24, 16], running_frac=0.6, queued_frac=0.3, depth=3)
    a = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue, st.priority, 3)
    inf = np.full(80, np.inf, np.float32)
    b = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue, st.priority, 3,
                    batch=np.full(80, 64, np.int32), iters=np.full(80, 1e4, np.float32), deadline=inf)
    assert a == b


@pytest.mark.parametrize("seed", [1, 2])
def test_deadline_invariants_on_random_states(seed):
    counts = [1, 2, 4, 8, 16, 32]
    thr = ss.synthetic_thr(seed, 80, 3, counts)
    st = ss.random_state(seed, thr, counts, [40, 24, 16], running_frac=0.6, queued_frac=0.3, depth=4)
    B, N, D = ss.deadlines(seed, st.thr)
    r = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue, st.priority,
                    st.depth, batch=B, iters=N, deadline=D)
    for q, j in enumerate(st.queue):
        if r["launched"][q]:       # every launch meets its deadline
            v = float(st.thr[j, r["alloc_type"][j], r["alloc_count"][j]])
            assert float(B[j]) * float(N[j]) / v <= float(D[j])
    for j in range(st.n_jobs):      # every moved running job sits on an open grid
        if st.alloc_type[j] >= 0 and r["alloc_count"][j] != st.alloc_count[j]:
            v = float(st.thr[j, r["alloc_type"][j], r["alloc_count"][j]])
            assert float(B[j]) * float(N[j]) / v <= float(D[j])


# ---------------------------------------------------------------- Eq. 7 (S9)
# rho = B N / (thr n): the finish-time-fairness ratio of a job on n GPUs.

def test_fairness_scale_up_helps_the_worst_job():
    # job 0: B N = 100 at 10 samples/s on 1 GPU -> rho 10; job 1: B N = 20 at 1/s -> rho 20.
    # Eq. 5 moves job 0 first (gain 9/GPU to 2 GPUs vs job 1's 0.5); Eq. 7 moves job 1, the
    # worst, to the count with its least rho: 2 GPUs 20 / 3 = 6.67, 4 GPUs 20 / 7.2 = 2.78.
    thr = _thr({0: [[10, 19, 36]], 1: [[1, 1.5, 1.8]]})
    kw = dict(batch=[1, 1], iters=[100.0, 20.0])
    r = so.schedule(thr, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 1)
    assert r["alloc_count"] == [1, 0]
    r = so.schedule(thr, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 1, objective="fairness", **kw)
    assert r["alloc_count"] == [0, 2] and r["moves"] == [0, 0, 1] and r["free"] == [1]
    # depth 3: then job 0 (rho 10) takes the last GPU (100 / 38 = 2.63); job 1 (2.78) is now
    # the worst but at its largest count, and nothing is free: the third search finds nothing
    r = so.schedule(thr, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 3, objective="fairness", **kw)
    assert r["alloc_count"] == [1, 2] and r["moves"] == [0, 0, 2] and r["free"] == [0]
    assert r["decisions"] == 3


def test_fairness_scale_down_takes_from_the_least_harmed():
    # 8 GPUs all busy, job 2 needs 1.  Eq. 5 shrinks job 0 (loses 0.5/GPU vs job 1's 0.6/GPU);
    # Eq. 7 shrinks the job whose rho after the step is smallest: job 1, 137.6 / (40 * 2) = 1.720
    # against job 0's 100 / (29 * 2) = 1.724 -- though job 1's rho before the step is the larger
    # (137.6 / (41.2 * 4) = 0.835 vs 100 / (30 * 4) = 0.833).  Job 2 then launches on 2 GPUs.
    thr = _thr({0: [[10, 29, 30]], 1: [[5, 40, 41.2]], 2: [[1, 2, 3]]})
    args = ([1, 2, 4], [8], [0, 0, -1], [2, 2, 0], [2], [0], 4)
    r = so.schedule(thr, *args)
    assert r["alloc_count"][:2] == [1, 2]
    r = so.schedule(thr, *args, batch=[1, 1, 1], iters=[100.0, 137.6, 5.0], objective="fairness")
    assert r["alloc_count"] == [2, 1, 1] and r["alloc_type"] == [0, 0, 0]
    assert r["launched"] == [1] and r["moves"] == [1, 1, 0] and r["decisions"] == 4


def test_fairness_target_ties_go_to_the_smaller_count():
    # thr * n = 4, 6, 6: rho on 2 and on 4 GPUs is exactly 1 (B N = 6): the smaller count
    thr = _thr({0: [[4, 3, 1.5]]})
    r = so.schedule(thr, [1, 2, 4], [4], [0], [0], [], [], 1, batch=[2], iters=[3.0], objective="fairness")
    assert r["alloc_count"] == [1] and r["moves"] == [0, 0, 1]


def test_fairness_moves_only_when_rho_falls_and_ties_go_to_the_lower_job():
    # no work left (N = 0): rho is 0 on every grid, nothing improves, nothing moves
    thr = _thr({0: [[1, 2, 4]], 1: [[1, 2, 4]]})
    r = so.schedule(thr, [1, 2, 4], [8], [0, 0], [0, 0], [], [], 4, batch=[1, 1], iters=[0.0, 0.0],
                    objective="fairness")
    assert r["alloc_count"] == [0, 0] and r["moves"] == [0, 0, 0]
    # equal rho (B N = 8 on 1 GPU at 1/s): job 0 moves first, to 4 GPUs (rho 0.5); one GPU is
    # left, so job 1 goes to 2 GPUs (rho 2) -- 4 would need 3 more
    r = so.schedule(thr, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 4, batch=[1, 1], iters=[8.0, 8.0],
                    objective="fairness")
    assert r["alloc_count"] == [2, 1] and r["moves"] == [0, 0, 2]


def test_fairness_with_a_deadline_scales_up_within_it():
    # the tie of the previous test broken by a deadline: job 1 may only finish in time on 4 GPUs
    # (8 / 4 = 2 s <= 2.5 s), which does not fit after job 0's move; with 6 free it would
    thr = _thr({0: [[1, 2, 4]], 1: [[1, 2, 4]]})
    kw = dict(batch=[1, 1], iters=[8.0, 8.0], deadline=[1e9, 2.5], objective="fairness")
    r = so.schedule(thr, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 4, **kw)
    assert r["alloc_count"] == [2, 0] and r["moves"] == [0, 0, 1]


def test_fairness_needs_work_and_checks_the_objective():
    thr = _thr({0: [[1, 2]], 1: [[1, 2]]})
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [4], [-1, -1], [0, 0], [0], [0], 1, objective="fairness")
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [4], [-1, -1], [0, 0], [0], [0], 1, batch=[1, 1], objective="fairness")
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [4], [-1, -1], [0, 0], [0], [0], 1, objective="makespan")
    with pytest.raises(ValueError):
        so.schedule(thr, [1, 2], [4], [-1, -1], [0, 0], [0], [0], 1, batch=[1, 1], iters=[-1.0, 1.0],
                    objective="fairness")


def _rho_all(st, r, B, N):
    out = []
    for j in range(st.n_jobs):
        g = r["alloc_type"][j]
        if g >= 0:
            v = float(st.thr[j, g, r["alloc_count"][j]])
            out.append(float(B[j]) * float(N[j]) / (v * st.counts[r["alloc_count"][j]]) if v > 0 else np.inf)
    return out


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_fairness_invariants_on_random_states(seed):
    counts = [1, 2, 4, 8, 16, 32]
    thr = ss.synthetic_thr(seed, 80, 3, counts)
    st = ss.random_state(seed, thr, counts, [40, 24, 16], running_frac=0.6, queued_frac=0.3, depth=4)
    B, N, _ = ss.deadlines(seed, st.thr)
    r = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue, st.priority,
                    st.depth, batch=B, iters=N, objective="fairness")
    used = np.zeros(3, np.int64)
    for j in range(st.n_jobs):
        g = r["alloc_type"][j]
        if g >= 0:
            used[g] += counts[r["alloc_count"][j]]
            if st.alloc_type[j] >= 0:
                assert g == st.alloc_type[j]
    assert list(used + np.asarray(r["free"])) == list(st.capacity) and min(r["free"]) >= 0
    # without a queue every move lowers the rho of one job: the largest rho never rises
    r0 = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, [], [], 1,
                     batch=B, iters=N, objective="fairness")
    before = _rho_all(st, dict(alloc_type=list(st.alloc_type), alloc_count=list(st.alloc_count)), B, N)
    prev = max(before)
    for d in range(1, 6):
        rd = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, [], [], d,
                         batch=B, iters=N, objective="fairness")
        now = max(_rho_all(st, rd, B, N))
        assert now <= prev
        prev = now
    assert r0["moves"][2] in (0, 1)
