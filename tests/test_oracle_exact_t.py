"""How far the balanced partition is from the partition that minimises the
whole iteration time (the exact-T partition), by brute force on the tiny
workload (L = 12: every cut vector of every plan priced by the oracle).

The balanced rule (reading R11) picks the split with the least slowest stage
and prices the plan on it; the full iteration time (Sec. 3.4, 1F1B) also has
the p2p sum and the largest DP all-reduce, so another split can be faster.
Pins: for every plan the brute-force optimum is never above the balanced or
the memory-constrained price, equals them at pp = 1, and a plan is feasible
under the memory-constrained rule exactly when some split fits memory.  The
gaps are printed (CPU only)."""
import dataclasses
import itertools

import numpy as np
import pytest

from paper_2403_16125_amd import workloads as wl


def _plans(w, j, g, n):
    """(dp, tp, pp, m) of cell (j, g, n): dp tp pp = n, tp divides n and the
    node size, pp <= L, dp m divides the global batch (Eq. 1)."""
    L = w.layers(j)
    Bg = int(w.batch[j])
    gpn = int(w.gpus_per_node[g])
    out = []
    for tp in range(1, n + 1):
        if n % tp or gpn % tp:
            continue
        for pp in range(1, min(n // tp, L) + 1):
            if (n // tp) % pp:
                continue
            dp = n // (tp * pp)
            for m in w.m_values:
                if Bg % (dp * int(m)) == 0:
                    out.append((dp, tp, pp, int(m)))
    return out


@pytest.mark.parametrize("mem_scale", [1.0, 0.05])
def test_exact_t_by_brute_force_on_tiny(oracle, mem_scale):
    # mem_scale 0.05: GPU memory cut to 2 / 4 GB, so that the limit binds for most plans
    w = wl.make("tiny")
    w = dataclasses.replace(w, mem=(w.mem * mem_scale).astype(np.float32))
    n_fit = 0
    gaps, cell_gaps, cell_gaps_mem = [], [], []
    n_plans = n_opt = 0
    for j in range(w.n_jobs):
        L = w.layers(j)
        for g in range(w.n_types):
            for ci, n in enumerate(int(c) for c in w.counts):
                kap = float(w.kappa[0][g * w.n_counts + ci])
                best_bal = best_mem = best_exact = np.inf
                for dp, tp, pp, m in _plans(w, j, g, n):
                    bal = oracle.eval_plan(w, j, g, n, kap, dp, tp, pp, m)
                    mem = oracle.eval_plan(w, j, g, n, kap, dp, tp, pp, m, rule=1)
                    exact = np.inf
                    for cuts in itertools.combinations(range(1, L), pp - 1):
                        e = oracle.eval_plan(w, j, g, n, kap, dp, tp, pp, m, cuts=list(cuts))
                        if e["feasible"]:
                            exact = min(exact, e["T"])
                    n_plans += 1
                    n_fit += bool(np.isfinite(exact))
                    assert mem["feasible"] == np.isfinite(exact)       # rule 1 finds a fitting split iff one exists
                    for r in (bal, mem):
                        if r["feasible"]:
                            assert exact <= r["T"] * (1 + 1e-12)
                            if pp == 1:
                                assert exact == r["T"]
                    if bal["feasible"]:
                        gaps.append(bal["T"] / exact - 1.0)
                        n_opt += bal["T"] <= exact * (1 + 1e-12)
                        best_bal = min(best_bal, bal["T"])
                    if mem["feasible"]:
                        best_mem = min(best_mem, mem["T"])
                    best_exact = min(best_exact, exact)
                if np.isfinite(best_bal):
                    cell_gaps.append(best_bal / best_exact - 1.0)
                if np.isfinite(best_mem):
                    cell_gaps_mem.append(best_mem / best_exact - 1.0)
    gaps, cell_gaps, cell_gaps_mem = np.asarray(gaps), np.asarray(cell_gaps), np.asarray(cell_gaps_mem)
    print(f"[exact-T] tiny, memory x{mem_scale}: {n_plans} plans, {n_fit} with a split that fits, "
          f"{len(gaps)} feasible under the balanced rule; balanced split "
          f"optimal for {n_opt} ({100 * n_opt / len(gaps):.1f} %); plan gap mean {100 * gaps.mean():.3f} % "
          f"max {100 * gaps.max():.3f} %; best-plan gap per cell mean {100 * cell_gaps.mean():.3f} % "
          f"max {100 * cell_gaps.max():.3f} % over {len(cell_gaps)} cells; memory rule's best plan: mean "
          f"{100 * cell_gaps_mem.mean():.3f} % max {100 * cell_gaps_mem.max():.3f} % over {len(cell_gaps_mem)} cells")
    assert (gaps >= -1e-12).all() and (cell_gaps >= -1e-12).all() and (cell_gaps_mem >= -1e-12).all()
    assert n_plans > 100 and len(cell_gaps) > 5
