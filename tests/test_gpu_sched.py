"""Parity of the HIP scheduling step (arena_schedule) with the CPU oracle of
Algorithm 1 under the throughput objective (Sec. 3.5, Eq. 5), the deadline
constraint (Eq. 6) and the finish-time fairness objective (Eq. 7), through the
C ABI.

Both sides take every decision in float64 from the same float32 throughput
matrix, so the agreement is exact: the new allocation of every job, which
queued jobs launched, and the move counts.  Inputs are seeded synthetic
throughput curves and cluster states (sched_states)."""
import numpy as np
import pytest

from oracle import scheduler_oracle as so
from paper_2403_16125_amd import sched_states as ss

def _gpu(st, ddl=None, objective="throughput"):
    from paper_2403_16125_amd import arena
    s = arena.Scheduler(st.thr, st.counts, st.capacity, objective=objective)
    if ddl is not None:
        s.set_deadlines(*ddl)
    try:
        s.load_state(st.alloc_type, st.alloc_count, st.queue, st.priority)
        s.step(st.depth)
        return s.results()
    finally:
        s.close()


def _check(st, ddl=None, objective="throughput"):
    print(f"schedule: J={st.n_jobs} T={st.thr.shape[1]} NC={st.thr.shape[2]} Q={len(st.queue)} "
          f"D={st.depth} deadlines={ddl is not None and ddl[2] is not None} objective={objective}", flush=True)
    kw = {} if ddl is None else dict(batch=ddl[0], iters=ddl[1], deadline=ddl[2])
    want = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue,
                       st.priority, st.depth, objective=objective, **kw)
    got = _gpu(st, ddl, objective)
    assert got["status"] == 0
    assert got["moves"] == want["moves"]
    assert got["decisions"] == want["decisions"]
    assert list(got["launched"]) == want["launched"]
    bad = np.nonzero((got["alloc_type"] != np.asarray(want["alloc_type"])) |
                     (got["alloc_count"] != np.asarray(want["alloc_count"])))[0]
    assert len(bad) == 0, f"{len(bad)} jobs differ, first {bad[:8]}"
    return want


def _state(thr_rows, counts, capacity, alloc_type, alloc_count, queue, priority, depth):
    J = max(thr_rows) + 1
    T = len(next(iter(thr_rows.values())))
    thr = np.zeros((J, T, len(counts)), np.float32)
    for j, r in thr_rows.items():
        thr[j] = np.asarray(r, np.float32)
    return ss.SchedState(thr=thr, counts=np.asarray(counts, np.int32),
                         capacity=np.asarray(capacity, np.int32),
                         alloc_type=np.asarray(alloc_type, np.int32),
                         alloc_count=np.asarray(alloc_count, np.int32),
                         queue=np.asarray(queue, np.int32), priority=np.asarray(priority, np.int32),
                         depth=int(depth))


HAND = {
    "launch": ({0: [[10, 18, 30], [12, 20, 25]]}, [1, 2, 4], [2, 4], [-1], [0], [0], [0], 4),
    "launch_tie": ({0: [[10, 20, 20], [5, 20, 20]]}, [1, 2, 4], [4, 4], [-1], [0], [0], [0], 4),
    "scale_down": ({0: [[0, 50, 80]], 1: [[10, 19, 0]], 2: [[3, 20, 0]]}, [1, 2, 4], [4],
                   [-1, 0, 0], [0, 1, 1], [0], [0], 4),
    "rollback": ({0: [[0, 50, 80]], 1: [[10, 19, 0]], 2: [[3, 20, 0]]}, [1, 2, 4], [4],
                 [-1, 0, 0], [0, 1, 1], [0], [0], 1),
    "usable_types": ({0: [[0, 0], [0, 40]], 1: [[10, 11], [0, 0]], 2: [[0, 0], [5, 30]]}, [1, 2],
                     [2, 3], [-1, 0, 1], [0, 1, 1], [0], [0], 4),
    "priority": ({0: [[0, 9]], 1: [[5, 8]], 2: [[0, 7]], 3: [[4, 0]]}, [1, 2], [2], [-1] * 4,
                 [0] * 4, [0, 1, 2, 3], [0, 0, 1, 1], 4),
    "scale_up": ({0: [[5, 9, 16, 20]], 1: [[4, 10, 19, 30]]}, [1, 2, 4, 8], [8], [0, 0], [1, 1],
                 [], [], 8),
    "scale_up_best_step": ({0: [[10, 11, 40]]}, [1, 2, 4], [4], [0], [0], [], [], 4),
    "scale_down_per_gpu": ({0: [[0, 50, 80]], 1: [[5, 20, 30]], 2: [[2, 10, 0]]}, [1, 2, 4], [6],
                           [-1, 0, 0], [0, 2, 1], [0], [0], 4),
    "allowance": ({0: [[0, 0, 50]], 1: [[10, 0, 0]]}, [1, 2, 4], [2], [-1, -1], [0, 0], [0, 1], [1, 1], 4),
}


@pytest.mark.gpu
@pytest.mark.parametrize("name", sorted(HAND))
def test_hand_cases(name):
    _check(_state(*HAND[name]))


@pytest.mark.gpu
def test_hand_case_values():
    # the GPU reproduces the hand-derived outcomes the oracle is pinned to
    got = _gpu(_state(*HAND["scale_down"]))
    assert list(got["alloc_count"]) == [1, 0, 0] and got["moves"] == [2, 1, 0]
    got = _gpu(_state(*HAND["rollback"]))
    assert list(got["alloc_count"]) == [0, 1, 1] and list(got["alloc_type"]) == [-1, 0, 0]
    got = _gpu(_state(*HAND["scale_up"]))
    assert list(got["alloc_count"]) == [2, 2] and got["moves"] == [0, 0, 2]


# (seed, jobs, types, counts, capacity, running share, queued share, classes, depth, max count)
RANDOM = [
    (1, 60, 3, [1, 2, 4, 8, 16, 32], [40, 24, 16], 0.5, 0.3, 3, 4, None),
    (2, 60, 3, [1, 2, 4, 8, 16, 32], [40, 24, 16], 0.9, 0.1, 2, 1, None),
    (3, 300, 4, [1, 2, 3, 4, 6, 8, 12, 16], [64, 32, 32, 16], 0.7, 0.2, 3, 8, 8),
    (4, 1100, 5, [1, 2, 4, 8, 16, 24, 32, 48, 64, 96, 128], [256, 128, 128, 64, 64], 0.6, 0.1, 4,
     16, 16),
    (5, 1500, 8, [1, 2, 4, 8, 16, 32, 64], [96] * 8, 0.3, 0.3, 1, 3, 4),
    (6, 777, 6, [1, 2, 4, 8, 16, 32, 64, 128], [200, 0, 150, 90, 60, 30], 0.8, 0.15, 3, 256, 32),
    (7, 64, 2, [1, 2, 4, 8], [0, 0], 0.0, 0.5, 2, 3, None),            # no GPUs at all
    (8, 200, 3, [2, 4, 8], [512, 512, 512], 0.2, 0.6, 3, 2, None),     # roomy cluster: scale-ups
]


@pytest.mark.gpu
@pytest.mark.parametrize("case", RANDOM, ids=[f"seed{c[0]}_J{c[1]}" for c in RANDOM])
def test_random_states(case):
    seed, J, T, counts, cap, rf, qf, ncls, depth, mc = case
    thr = ss.synthetic_thr(seed, J, T, counts)
    st = ss.random_state(seed, thr, counts, cap, running_frac=rf, queued_frac=qf, n_classes=ncls,
                         depth=depth, max_count=mc)
    _check(st)


def test_random_states_cover_every_move():
    # the random cases above exercise kept scale-downs, launches, scale-ups and
    # jobs left queued (CPU only: checked on the oracle's outcome)
    seen = np.zeros(4, np.int64)
    for seed, J, T, counts, cap, rf, qf, ncls, depth, mc in RANDOM:
        thr = ss.synthetic_thr(seed, J, T, counts)
        st = ss.random_state(seed, thr, counts, cap, running_frac=rf, queued_frac=qf,
                             n_classes=ncls, depth=depth, max_count=mc)
        r = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue,
                        st.priority, st.depth)
        seen[:3] += r["moves"]
        seen[3] += len(st.queue) - sum(r["launched"])
    assert (seen > 0).all(), seen


@pytest.mark.gpu
def test_full_round_matrix():
    # the state the benchmark times: 16384 jobs x 8 types x 131 counts, a
    # 1280-GPU cluster, search depth 3
    want = _check(ss.full_round())
    assert want["moves"][1] > 0


@pytest.mark.gpu
@pytest.mark.parametrize("n_run", [4096, 5000])
def test_many_running_jobs(n_run):
    # running jobs beyond what the kernel keeps in its LDS list (5000), and a
    # list that is full at the start (4096) so that the first launch of the
    # step overflows it: the rest of the step scans every job
    counts = [1, 2, 4, 8]
    J = n_run + 150
    thr = ss.synthetic_thr(41, J, 2, counts)
    at = np.full(J, -1, np.int32)
    ac = np.zeros(J, np.int32)
    used = np.zeros(2, np.int64)
    for j in range(n_run):
        g = j % 2
        c = int(np.argmax(thr[j, g] > 0))     # smallest count with throughput > 0
        assert thr[j, g, c] > 0
        at[j], ac[j] = g, c
        used[g] += counts[c]
    cap = (used + 64).astype(np.int32)
    queue = np.arange(n_run, J, dtype=np.int32)
    st = ss.SchedState(thr=thr, counts=np.asarray(counts, np.int32), capacity=cap, alloc_type=at,
                       alloc_count=ac, queue=queue, priority=np.zeros(len(queue), np.int32),
                       depth=4)
    want = _check(st)
    assert want["moves"][0] > 0 and want["moves"][1] > 0


@pytest.mark.gpu
def test_empty_queue_and_no_jobs():
    st = _state({0: [[1, 2]], 1: [[3, 4]]}, [1, 2], [4], [0, -1], [0, 0], [], [], 2)
    _check(st)
    from paper_2403_16125_amd import arena
    s = arena.Scheduler(np.zeros((0, 2, 3), np.float32), [1, 2, 4], [4, 4])
    try:
        s.load_state(np.zeros(0, np.int32), np.zeros(0, np.int32), [], [])
        s.step(1)
        r = s.results()
        assert r["status"] == 0 and r["moves"] == [0, 0, 0]
    finally:
        s.close()


@pytest.mark.gpu
def test_largest_shapes():
    # 64 types x 512 counts (the limits), depth 256
    counts = list(range(1, 513))
    thr = ss.synthetic_thr(21, 40, 64, counts)
    st = ss.random_state(21, thr, counts, [300] * 64, running_frac=0.6, queued_frac=0.4,
                         n_classes=2, depth=256, max_count=64)
    _check(st)


@pytest.mark.parametrize("kind", ["over_capacity", "queued_running", "listed_twice", "bad_type",
                                  "bad_count", "negative_class", "queue_out_of_range"])
@pytest.mark.gpu
def test_bad_states_leave_everything_unchanged(kind):
    from paper_2403_16125_amd import arena
    base = dict(at=[0, -1, -1], ac=[1, 0, 0], q=[1, 2], p=[0, 1], cap=[4])
    if kind == "over_capacity":
        base.update(ac=[2, 0, 0], cap=[3])
    elif kind == "queued_running":
        base.update(q=[0, 2])
    elif kind == "listed_twice":
        base.update(q=[1, 1])
    elif kind == "bad_type":
        base.update(at=[1, -1, -1])
    elif kind == "bad_count":
        base.update(ac=[3, 0, 0])
    elif kind == "negative_class":
        base.update(p=[0, -1])
    elif kind == "queue_out_of_range":
        base.update(q=[1, 3])
    thr = np.full((3, 1, 3), 5.0, np.float32)
    s = arena.Scheduler(thr, [1, 2, 4], base["cap"])
    try:
        s.load_state(base["at"], base["ac"], base["q"], base["p"])
        s.launched.fill_(-7)
        s.step(2)
        r = s.results()
        assert r["status"] == (1 if kind == "over_capacity" else 2)
        assert list(r["alloc_type"]) == base["at"] and list(r["alloc_count"]) == base["ac"]
        assert (r["launched"] == -7).all()
    finally:
        s.close()


@pytest.mark.gpu
def test_repeated_steps_on_device_state():
    # steps chain on the device-resident allocation: each step equals the
    # oracle's step from the state the previous oracle step left; only the
    # queue (the jobs still waiting) is uploaded between steps
    counts = [1, 2, 4, 8, 16]
    thr = ss.synthetic_thr(31, 400, 4, counts)
    st = ss.random_state(31, thr, counts, [64, 48, 32, 16], running_frac=0.7, queued_frac=0.25,
                         n_classes=3, depth=3, max_count=8)
    from paper_2403_16125_amd import arena
    s = arena.Scheduler(st.thr, st.counts, st.capacity)
    try:
        at, ac = st.alloc_type.copy(), st.alloc_count.copy()
        queue, prio = list(st.queue), list(st.priority)
        s.load_state(at, ac, queue, prio)
        for step in range(4):
            want = so.schedule(st.thr, counts, st.capacity, at, ac, queue, prio, st.depth)
            s.step(st.depth)
            got = s.results()
            assert got["status"] == 0 and got["moves"] == want["moves"], step
            assert list(got["alloc_type"]) == want["alloc_type"], step
            assert list(got["alloc_count"]) == want["alloc_count"], step
            at = np.asarray(want["alloc_type"], np.int32)
            ac = np.asarray(want["alloc_count"], np.int32)
            keep = [k for k in range(len(queue)) if not want["launched"][k]]
            queue, prio = [queue[k] for k in keep], [prio[k] for k in keep]
            s.load_queue(queue, prio)
    finally:
        s.close()


# ---------------------------------------------------------------- deadlines (Eq. 6)

DDL_HAND = {
    "launch_gate": (({0: [[10, 18, 30]]}, [1, 2, 4], [2], [-1], [0], [0], [0], 4),
                    ([10], [30.0], [12.0])),
    "launch_open": (({0: [[10, 18, 30]]}, [1, 2, 4], [4], [-1], [0], [0], [0], 4),
                    ([10], [30.0], [12.0])),
    "scale_down_protected": (({0: [[0, 50, 80]], 1: [[10, 19, 0]], 2: [[3, 20, 0]]}, [1, 2, 4], [4],
                              [-1, 0, 0], [0, 1, 1], [0], [0], 4), ([1, 1, 1], [1.0, 100.0, 1.0], [1e9, 6.0, 1e9])),
    "scale_up_steered": (({0: [[1, 2, 4]]}, [1, 2, 4], [4], [0], [0], [], [], 1), ([1], [10.0], [3.0])),
    "met_exactly": (({0: [[10, 20]]}, [1, 2], [2], [-1], [0], [0], [0], 4), ([4], [10.0], [2.0])),
}


@pytest.mark.gpu
@pytest.mark.parametrize("name", sorted(DDL_HAND))
def test_deadline_hand_cases(name):
    args, ddl = DDL_HAND[name]
    _check(_state(*args), tuple(np.asarray(v) for v in ddl))


@pytest.mark.gpu
@pytest.mark.parametrize("case", RANDOM[:6], ids=[f"seed{c[0]}_J{c[1]}" for c in RANDOM[:6]])
def test_deadline_random_states(case):
    seed, J, T, counts, cap, rf, qf, ncls, depth, mc = case
    thr = ss.synthetic_thr(seed, J, T, counts)
    st = ss.random_state(seed, thr, counts, cap, running_frac=rf, queued_frac=qf, n_classes=ncls,
                         depth=depth, max_count=mc)
    _check(st, ss.deadlines(seed, st.thr))


@pytest.mark.gpu
def test_deadline_full_round():
    st = ss.full_round()
    _check(st, ss.deadlines(11, st.thr, slack=(0.9, 4.0)))


@pytest.mark.gpu
def test_infinite_deadlines_change_nothing():
    counts = [1, 2, 4, 8, 16]
    thr = ss.synthetic_thr(12, 300, 4, counts)
    st = ss.random_state(12, thr, counts, [64, 48, 32, 16], running_frac=0.7, queued_frac=0.25, depth=3)
    a = _gpu(st)
    b = _gpu(st, (np.full(300, 128, np.int32), np.full(300, 1e4, np.float32), np.full(300, np.inf, np.float32)))
    assert a["moves"] == b["moves"] and (a["alloc_count"] == b["alloc_count"]).all()
    assert (a["launched"] == b["launched"]).all()


@pytest.mark.gpu
@pytest.mark.parametrize("bad", ["batch", "iters", "deadline"])
def test_bad_deadline_values_leave_everything_unchanged(bad):
    from paper_2403_16125_amd import arena
    thr = np.full((3, 1, 3), 5.0, np.float32)
    B, N, D = np.full(3, 8, np.int32), np.full(3, 10.0, np.float32), np.full(3, 100.0, np.float32)
    if bad == "batch":
        B[1] = 0
    elif bad == "iters":
        N[2] = np.nan
    else:
        D[0] = -1.0
    s = arena.Scheduler(thr, [1, 2, 4], [4], batch=B, iters=N, deadline=D)
    try:
        s.load_state([0, -1, -1], [1, 0, 0], [1, 2], [0, 1])
        s.launched.fill_(-7)
        s.step(2)
        r = s.results()
        assert r["status"] == 2
        assert list(r["alloc_type"]) == [0, -1, -1] and list(r["alloc_count"]) == [1, 0, 0]
        assert (r["launched"] == -7).all()
    finally:
        s.close()


# ---------------------------------------------------------------- finish-time fairness (Eq. 7)

FAIR_HAND = {
    "up_worst_first": (({0: [[10, 19, 36]], 1: [[1, 1.5, 1.8]]}, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 3),
                       ([1, 1], [100.0, 20.0], None)),
    "down_least_harmed": (({0: [[10, 29, 30]], 1: [[5, 40, 41.2]], 2: [[1, 2, 3]]}, [1, 2, 4], [8],
                           [0, 0, -1], [2, 2, 0], [2], [0], 4), ([1, 1, 1], [100.0, 137.6, 5.0], None)),
    "target_tie": (({0: [[4, 3, 1.5]]}, [1, 2, 4], [4], [0], [0], [], [], 1), ([2], [3.0], None)),
    "no_work_left": (({0: [[1, 2, 4]], 1: [[1, 2, 4]]}, [1, 2, 4], [8], [0, 0], [0, 0], [], [], 4),
                     ([1, 1], [0.0, 0.0], None)),
    "job_tie": (({0: [[1, 2, 4]], 1: [[1, 2, 4]]}, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 4),
                ([1, 1], [8.0, 8.0], None)),
    "with_deadline": (({0: [[1, 2, 4]], 1: [[1, 2, 4]]}, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 4),
                      ([1, 1], [8.0, 8.0], [1e9, 2.5])),
    "zero_throughput_running": (({0: [[0, 2, 4]], 1: [[1, 2, 4]]}, [1, 2, 4], [6], [0, 0], [0, 0], [], [], 2),
                                ([1, 1], [8.0, 8.0], None)),
}


def _fair_args(ddl):
    B, N, D = ddl
    return (np.asarray(B, np.int32), np.asarray(N, np.float32),
            None if D is None else np.asarray(D, np.float32))


@pytest.mark.gpu
@pytest.mark.parametrize("name", sorted(FAIR_HAND))
def test_fairness_hand_cases(name):
    args, ddl = FAIR_HAND[name]
    _check(_state(*args), _fair_args(ddl), "fairness")


@pytest.mark.gpu
def test_fairness_hand_case_values():
    # the GPU reproduces the hand-derived outcomes the oracle is pinned to
    args, ddl = FAIR_HAND["up_worst_first"]
    got = _gpu(_state(*args), _fair_args(ddl), "fairness")
    assert list(got["alloc_count"]) == [1, 2] and got["moves"] == [0, 0, 2] and got["decisions"] == 3
    args, ddl = FAIR_HAND["down_least_harmed"]
    got = _gpu(_state(*args), _fair_args(ddl), "fairness")
    assert list(got["alloc_count"]) == [2, 1, 1] and got["moves"] == [1, 1, 0]


@pytest.mark.gpu
@pytest.mark.parametrize("case", RANDOM, ids=[f"seed{c[0]}_J{c[1]}" for c in RANDOM])
def test_fairness_random_states(case):
    seed, J, T, counts, cap, rf, qf, ncls, depth, mc = case
    thr = ss.synthetic_thr(seed, J, T, counts)
    st = ss.random_state(seed, thr, counts, cap, running_frac=rf, queued_frac=qf, n_classes=ncls,
                         depth=depth, max_count=mc)
    B, N, D = ss.deadlines(seed, st.thr)
    _check(st, (B, N, None), "fairness")
    if seed <= 3:
        _check(st, (B, N, D), "fairness")


def test_fairness_random_states_cover_every_move():
    # CPU only: the fairness cases above exercise kept scale-downs, launches and scale-ups
    seen = np.zeros(3, np.int64)
    for seed, J, T, counts, cap, rf, qf, ncls, depth, mc in RANDOM:
        thr = ss.synthetic_thr(seed, J, T, counts)
        st = ss.random_state(seed, thr, counts, cap, running_frac=rf, queued_frac=qf,
                             n_classes=ncls, depth=depth, max_count=mc)
        B, N, _ = ss.deadlines(seed, st.thr)
        r = so.schedule(st.thr, st.counts, st.capacity, st.alloc_type, st.alloc_count, st.queue,
                        st.priority, st.depth, batch=B, iters=N, objective="fairness")
        seen += r["moves"]
    assert (seen > 0).all(), seen


@pytest.mark.gpu
def test_fairness_full_round():
    st = ss.full_round()
    B, N, D = ss.deadlines(11, st.thr, slack=(0.9, 4.0))
    want = _check(st, (B, N, None), "fairness")
    assert want["moves"][1] > 0
    _check(st, (B, N, D), "fairness")


@pytest.mark.gpu
def test_fairness_many_running_jobs():
    # more running jobs than the kernel's LDS list holds: the scan path
    counts = [1, 2, 4, 8]
    J = 5150
    thr = ss.synthetic_thr(43, J, 2, counts)
    at = np.full(J, -1, np.int32)
    ac = np.zeros(J, np.int32)
    used = np.zeros(2, np.int64)
    for j in range(5000):
        g = j % 2
        c = int(np.argmax(thr[j, g] > 0))
        at[j], ac[j] = g, c
        used[g] += counts[c]
    cap = (used + 64).astype(np.int32)
    queue = np.arange(5000, J, dtype=np.int32)
    st = ss.SchedState(thr=thr, counts=np.asarray(counts, np.int32), capacity=cap, alloc_type=at,
                       alloc_count=ac, queue=queue, priority=np.zeros(len(queue), np.int32), depth=4)
    B, N, _ = ss.deadlines(43, thr)
    want = _check(st, (B, N, None), "fairness")
    assert want["moves"][1] > 0


@pytest.mark.gpu
@pytest.mark.parametrize("bad", ["batch", "iters"])
def test_fairness_bad_values_leave_everything_unchanged(bad):
    from paper_2403_16125_amd import arena
    thr = np.full((3, 1, 3), 5.0, np.float32)
    B, N = np.full(3, 8, np.int32), np.full(3, 10.0, np.float32)
    if bad == "batch":
        B[1] = -2
    else:
        N[2] = np.inf
    s = arena.Scheduler(thr, [1, 2, 4], [4], batch=B, iters=N, objective="fairness")
    try:
        s.load_state([0, -1, -1], [1, 0, 0], [1, 2], [0, 1])
        s.launched.fill_(-7)
        s.step(2)
        r = s.results()
        assert r["status"] == 2
        assert list(r["alloc_type"]) == [0, -1, -1] and list(r["alloc_count"]) == [1, 0, 0]
        assert (r["launched"] == -7).all()
    finally:
        s.close()
