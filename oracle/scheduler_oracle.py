"""CPU oracle of one scheduling step over the throughput matrix.

TEST INFRASTRUCTURE ONLY: imported by tests/ and nothing on the product path.

Follows the event-driven scheduling of Sec. 3.5 (Algorithm 1) with the
throughput-maximisation objective of Eq. 5, written out with plain loops.
The paper leaves the inner steps open; the readings used here are:

S1  Queued jobs are visited in the given queue order (the caller sorts by
    priority class, smaller first).
S2  A job launches on the grid (type g, count n) with the highest throughput
    among grids with throughput > 0 and n <= the free GPUs of type g; ties go
    to the smaller count, then the lower type.  Jobs stay on one type
    (intra-job homogeneity, Sec. 3.5).
S3  If it cannot launch, the in-flight job whose scale-down loses the least
    throughput per GPU freed is scaled down (GetOptimalScaleDown): a job on a
    type where the queued job has some grid with throughput > 0 moves to the
    largest smaller count with throughput > 0; cost = (thr(n) - thr(n')) /
    (n - n') in float64 from the float32 matrix; ties go to the lower job id.
S4  Scale-downs repeat until the job launches or D of them were made; if it
    still cannot launch they are undone and the job stays queued.
S5  Priority rule of Algorithm 1: lam' starts above every class; a job that
    cannot launch sets lam' to its class if that is <= lam', and stops the
    visit if its class is > lam'.
S6  Then in-flight jobs are scaled up (GetOptimalScaleUp): each job's best
    move is to the larger count n' on its type with n' - n <= the free GPUs
    of the type and thr(n') > thr(n) that maximises (thr(n') - thr(n)) /
    (n' - n) (ties: the smaller n'); the job with the largest such gain moves
    (ties: the lower job id); at most D moves.

S8  Deadline constraint (Eq. 6), when per-job batch B_i, remaining
    iterations N_i and deadline DDL_i are given: a grid of throughput thr is
    open to job i only if thr > 0 and B_i N_i / thr <= DDL_i (float64).
    Every step above uses open grids only: launches (S2), the usable types
    and the scale-down target (S3: the largest smaller count still open) and
    scale-ups (S6: a larger open count).  A running job outside its deadline
    is not moved for it.

S9  Finish-time fairness objective (Eq. 7), when asked for, with per-job
    batch B_i and remaining iterations N_i (deadlines optional): the
    allocation indicator in the denominator is read as selecting the job's
    grid, and the resource measure Q of a grid as its GPU count, so a job
    running at throughput thr on n GPUs has rho = N_i T / n with T = B_i /
    thr, i.e. rho = B_i N_i / (thr n) in float64 (+inf at thr = 0).  The
    objective minimises the largest rho, so the two searches of Algorithm 1
    change their keys: GetOptimalScaleDown moves the job whose rho after
    its step down is smallest (same candidates as S3; ties: the lower job
    id); GetOptimalScaleUp takes, for each running job, the larger count
    within the free GPUs (and open, under S8) that minimises its rho (ties:
    the smaller count), kept only if that rho is below its current one, and
    moves the job whose current rho is largest (ties: the lower job id).
    Launches (S2) and everything else are unchanged.

Returns the new allocation, which queued jobs launched, the move counts
(scale-downs kept, launches, scale-ups) and the number of searches made
(launch, scale-down and scale-up: the decisions of the step).
"""
from __future__ import annotations


def _free(thr, counts, capacity, alloc_type, alloc_count):
    free = [int(c) for c in capacity]
    for j in range(len(alloc_type)):
        g = int(alloc_type[j])
        if g >= 0:
            free[g] -= int(counts[int(alloc_count[j])])
    return free


def _open(v, work, ddl):
    """S8: a grid of throughput v is open (work = B N; ddl None: no deadline)."""
    return v > 0.0 and (ddl is None or work / v <= ddl)


def launch_grid(thr_j, counts, free, work=0.0, ddl=None):
    """S2: best grid of one job under the free GPUs, or None."""
    best = None
    for g in range(len(free)):
        for c in range(len(counts)):
            v = float(thr_j[g][c])
            if _open(v, work, ddl) and int(counts[c]) <= free[g]:
                key = (-v, int(counts[c]), g)
                if best is None or key < best[0]:
                    best = (key, g, c)
    return None if best is None else (best[1], best[2])


def _rho(v, n, work):
    """S9: B N / (thr n) of a job with work B N at throughput v on n GPUs."""
    return work / (v * float(n)) if v > 0.0 else float("inf")


def scale_down_move(thr, counts, alloc_type, alloc_count, usable_types, dl=None, fair=False):
    """S3: (cost, job, new count index) of the cheapest scale-down, or None.
    dl(i) -> (work, deadline) of job i under S8 (deadline None: none); with
    fair (S9) the cost is the job's rho after the step."""
    best = None
    for i in range(len(alloc_type)):
        g = int(alloc_type[i])
        if g < 0 or g not in usable_types:
            continue
        work, ddl = dl(i) if dl else (0.0, None)
        c = int(alloc_count[i])
        c2 = c - 1
        while c2 >= 0 and not _open(float(thr[i][g][c2]), work, ddl):
            c2 -= 1
        if c2 < 0:
            continue
        if fair:
            cost = _rho(float(thr[i][g][c2]), int(counts[c2]), work)
        else:
            cost = (float(thr[i][g][c]) - float(thr[i][g][c2])) / float(int(counts[c]) - int(counts[c2]))
        if best is None or cost < best[0]:
            best = (cost, i, c2)
    return best


def scale_up_move(thr, counts, alloc_type, alloc_count, free, dl=None, fair=False):
    """S6: (gain, job, new count index) of the best scale-up, or None; with
    fair (S9): (current rho, job, new count index) of the job moved."""
    best = None
    for i in range(len(alloc_type)):
        g = int(alloc_type[i])
        if g < 0:
            continue
        work, ddl = dl(i) if dl else (0.0, None)
        c = int(alloc_count[i])
        n, t = int(counts[c]), float(thr[i][g][c])
        mine = None
        if fair:
            r0 = _rho(t, n, work)
            for c2 in range(c + 1, len(counts)):
                if int(counts[c2]) - n > free[g]:
                    break
                t2 = float(thr[i][g][c2])
                if _open(t2, work, ddl):
                    r2 = _rho(t2, int(counts[c2]), work)
                    if mine is None or r2 < mine[0]:
                        mine = (r2, c2)
            if mine is not None and mine[0] < r0 and (best is None or r0 > best[0]):
                best = (r0, i, mine[1])
            continue
        for c2 in range(c + 1, len(counts)):
            dn = int(counts[c2]) - n
            if dn > free[g]:
                break
            t2 = float(thr[i][g][c2])
            if t2 > t and _open(t2, work, ddl):
                gain = (t2 - t) / float(dn)
                if mine is None or gain > mine[0]:
                    mine = (gain, c2)
        if mine is not None and (best is None or mine[0] > best[0]):
            best = (mine[0], i, mine[1])
    return best


def schedule(thr, counts, capacity, alloc_type, alloc_count, queue, priority, depth,
             batch=None, iters=None, deadline=None, objective="throughput"):
    """One scheduling step (Algorithm 1, readings S1-S6; S8 with deadlines;
    S9 with objective "fairness", which needs batch and iters)."""
    alloc_type = [int(v) for v in alloc_type]
    alloc_count = [int(v) for v in alloc_count]
    for k in range(1, len(counts)):
        if not int(counts[k]) > int(counts[k - 1]):
            raise ValueError("counts must be strictly ascending")
    free = _free(thr, counts, capacity, alloc_type, alloc_count)
    if any(f < 0 for f in free):
        raise ValueError("the running jobs exceed the capacity")
    if len(set(int(j) for j in queue)) != len(queue) or any(alloc_type[int(j)] >= 0 for j in queue):
        raise ValueError("queued jobs must be distinct and not running")
    if any(int(p) < 0 for p in priority):
        raise ValueError("priority classes must be >= 0")
    if objective not in ("throughput", "fairness"):
        raise ValueError("objective must be 'throughput' or 'fairness'")
    fair = objective == "fairness"
    given = [v is not None for v in (batch, iters, deadline)]
    if fair and not (given[0] and given[1]):
        raise ValueError("the fairness objective needs batch and iters")
    if not fair and any(given) and not all(given):
        raise ValueError("give batch, iters and deadline together or none")
    dl = None
    if given[0] and given[1]:
        for i in range(len(alloc_type)):
            b, it = int(batch[i]), float(iters[i])
            if b <= 0 or not (it >= 0.0) or it == float("inf"):
                raise ValueError("bad deadline values")
            if deadline is not None and not (float(deadline[i]) > 0.0):
                raise ValueError("bad deadline values")
        if deadline is not None:
            dl = lambda i: (float(int(batch[i])) * float(iters[i]), float(deadline[i]))
        else:
            dl = lambda i: (float(int(batch[i])) * float(iters[i]), None)
    n_types = len(free)
    launched = [0] * len(queue)
    kept_down = launches = 0
    decisions = 0
    lam = max((int(p) for p in priority), default=0) + 1
    for q in range(len(queue)):
        j = int(queue[q])
        work, ddl = dl(j) if dl else (0.0, None)
        usable = {g for g in range(n_types) if any(_open(float(v), work, ddl) for v in thr[j][g])}
        log = []
        while True:
            grid = launch_grid(thr[j], counts, free, work, ddl)
            decisions += 1
            if grid is not None:
                g, c = grid
                alloc_type[j], alloc_count[j] = g, c
                free[g] -= int(counts[c])
                launched[q] = 1
                launches += 1
                kept_down += len(log)
                break
            if len(log) >= depth:
                grid = None
            else:
                mv = scale_down_move(thr, counts, alloc_type, alloc_count, usable, dl, fair)
                decisions += 1
                if mv is not None:
                    _, i, c2 = mv
                    g = alloc_type[i]
                    log.append((i, alloc_count[i]))
                    free[g] += int(counts[alloc_count[i]]) - int(counts[c2])
                    alloc_count[i] = c2
                    continue
            # no launch: undo the scale-downs, newest first
            for i, c_old in reversed(log):
                g = alloc_type[i]
                free[g] -= int(counts[c_old]) - int(counts[alloc_count[i]])
                alloc_count[i] = c_old
            break
        if not launched[q]:
            if int(priority[q]) <= lam:
                lam = int(priority[q])
            else:
                break
    ups = 0
    while ups < depth:
        mv = scale_up_move(thr, counts, alloc_type, alloc_count, free, dl, fair)
        decisions += 1
        if mv is None:
            break
        _, i, c2 = mv
        g = alloc_type[i]
        free[g] -= int(counts[c2]) - int(counts[alloc_count[i]])
        alloc_count[i] = c2
        ups += 1
    return dict(alloc_type=alloc_type, alloc_count=alloc_count, launched=launched,
                moves=[kept_down, launches, ups], free=free, decisions=decisions)
