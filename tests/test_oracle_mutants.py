"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of the oracle's C source (an in-flight
count off by one, the tensor degree dropped from the activations, a strict
memory limit, stages counted from the wrong end, the microbatch size missing
its m, a cut search that allows empty stages or completes with one stage too
few, a sum where the recursion takes a maximum), builds it with gcc into a
temporary library, and runs the pins of test_oracle_memory_partition.py
against it in a child process: some pin must fail (an assertion, or a crash
or time-out of the broken copy).  The unmodified copy, built the same way,
must pass them all.  The same is done for the balanced partition, the layer
costs, the plan price and the per-cell choice, the interpolated communication
latency, the proxy-plan planner's oracle and the scheduler's, each with its own
pins.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "arena_oracle.c")

MUTANTS = {
    "inflight_off_by_one": ("int inflight = M->m < pp - k ? M->m : pp - k;",
                            "int inflight = M->m < pp - k - 1 ? M->m : pp - k - 1;"),
    "activations_not_split_by_tp": ("(double)inflight * M->b * A / (double)M->tp;",
                                    "(double)inflight * M->b * A;"),
    "strict_memory_limit": ("return Mem <= M->mem;", "return Mem < M->mem;"),
    "stages_counted_from_the_front": ("if (!fits_sums(M, P, A, pp - t, pp)) continue;",
                                      "if (!fits_sums(M, P, A, t - 1, pp)) continue;"),
    "microbatch_size_without_m": ("M.b = b;\n        M.mem = ty->mem;",
                                  "M.b = (double)jb->Bg / (double)dp;\n        M.mem = ty->mem;"),
    # (checking the stage being closed as the next one is no mistake: the
    # smallest cut that leaves a splittable rest always gives a stage that
    # fits, so that check never binds; the completion test is what matters)
    "cut_search_allows_empty_stage": ("int c = prev + 1;", "int c = prev;"),
    "completion_one_stage_short": ("G[(pp - k) * L1 + c] <= W", "G[(pp - k - 1) * L1 + c] <= W"),
    "recursion_sum_not_max": ("double v = w > g ? w : g;", "double v = w + g;"),
}

RUNNER = r"""
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
from oracle import oracle as o
o._LIB = {lib!r}
o._lib = None
o.load()
import test_oracle_memory_partition as t
failed = []
def run(name, fn, *a):
    try:
        fn(*a)
    except AssertionError:
        failed.append(name)
for i, (case, want) in enumerate(t.HAND):
    run("hand%d" % i, t.test_hand_worked, o, case, want)
run("cell_weights", t.test_hand_cell_weights)
run("cell_activations", t.test_hand_cell_activations)
run("bruteforce", t.test_recursion_matches_bruteforce, o)
run("unlimited", t.test_unlimited_memory_is_the_unconstrained_partition, o)
run("kept_and_fit", t.test_fitting_unconstrained_partition_is_kept_and_results_fit, o)
run("monotone", t.test_more_memory_never_raises_the_bottleneck, o)
run("enumeration", t.test_small_cells_against_enumeration, o)
print("failed:", failed, flush=True)
sys.exit(1 if failed else 0)
"""


def _build(tmp_path, name, patch, source=SRC):
    src = open(source).read()
    if patch is not None:
        # the first occurrence: the function the pins exercise comes first
        # (the table-latency pricing repeats some of its lines further down)
        old, new = patch
        assert old in src, (name, old)
        src = src.replace(old, new, 1)
    c = tmp_path / f"{name}.c"
    c.write_text(src)
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
                    "-o", str(lib), str(c), "-lm"], check=True)
    return str(lib)


def _run_pins(lib):
    code = RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
    try:
        r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    except subprocess.TimeoutExpired:
        return None, "timed out"
    return r.returncode, (r.stdout + r.stderr)[-2000:]


def test_unmodified_copy_passes(tmp_path):
    lib = _build(tmp_path, "control", None)
    rc, out = _run_pins(lib)
    assert rc == 0, out
    rc, out = _run_pin_files(lib)
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    rc, out = _run_pins(_build(tmp_path, name, MUTANTS[name]))
    assert rc != 0, f"mistake {name} survived every pin: {out}"


# Mistakes in the balanced partition, the layer costs, the plan price and the
# per-cell choice, against the pins of test_oracle_partition.py and
# test_oracle_pricing.py (run by pytest in a child process on the copy).
CORE_MUTANTS = {
    "tp_comm_without_kappa": ("v += kappa * 8.0 * (double)(tp - 1) / (double)tp * (double)jb->x[l] / ty->bw_intra;",
                              "v += 8.0 * (double)(tp - 1) / (double)tp * (double)jb->x[l] / ty->bw_intra;"),
    "all_to_all_only_with_tp": ("if (dp * tp > 1)", "if (tp > 1)"),
    "p2p_of_the_next_layer": ("p2p = kappa * 2.0 * b * (double)jb->x[hi - 1] / B_pp;",
                              "p2p = kappa * 2.0 * b * (double)jb->x[hi] / B_pp;"),
    "allreduce_factor_halved": ("AR = kappa * 2.0 * (double)(dp - 1)", "AR = kappa * (double)(dp - 1)"),
    "pricing_inflight_off_by_one": ("int inflight = m < pp - k ? m : pp - k;",
                                    "int inflight = m < pp - k - 1 ? m : pp - k - 1;"),
    "steady_state_m_microbatches": ("r.T = fill + (double)(m - 1) * w_max + ar_max;",
                                    "r.T = fill + (double)m * w_max + ar_max;"),
    "pipeline_link_strict": ("double B_pp = (n <= ty->gpn)", "double B_pp = (n < ty->gpn)"),
    "dp_link_ignores_divisibility": ("(grp <= ty->gpn && ty->gpn % grp == 0)", "(grp <= ty->gpn)"),
    "recursion_skips_first_split": ("for (int j = k - 1; j <= i - 1; ++j)", "for (int j = k; j <= i - 1; ++j)"),
    "canonical_cut_tie_wrong_way": ("while (c < next - 1 && seg(U, c, next) > W) ++c;",
                                    "while (c < next - 1 && seg(U, c, next) >= W) ++c;"),
    "tie_window_strict": ("if (!cand[i].feasible || !(cand[i].T <= lim)) continue;",
                          "if (!cand[i].feasible || !(cand[i].T < lim)) continue;"),
    "key_tp_before_pp": ("if (a->pp != b->pp) return a->pp < b->pp;", "if (a->tp != b->tp) return a->tp < b->tp;"),
    "admissibility_ignores_dp": ("if (jb.Bg % (dp * m) != 0) continue;", "if (jb.Bg % m != 0) continue;"),
    "weights_counted_twice_not_four_times": ("double Mem = 4.0 * Pk / (double)tp", "double Mem = 2.0 * Pk / (double)tp"),
}


def _run_pin_files(lib):
    env = dict(os.environ, ARENA_ORACLE_LIB=lib)
    files = [os.path.join(ROOT, "tests", f) for f in ("test_oracle_partition.py", "test_oracle_pricing.py")]
    try:
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                            "-p", "no:xdist"] + files, capture_output=True, text=True, timeout=300, env=env,
                           cwd=ROOT)
    except subprocess.TimeoutExpired:
        return None, "timed out"
    return r.returncode, (r.stdout + r.stderr)[-2000:]


@pytest.mark.parametrize("name", sorted(CORE_MUTANTS))
def test_planted_core_mistake_is_caught(tmp_path, name):
    rc, out = _run_pin_files(_build(tmp_path, name, CORE_MUTANTS[name]))
    assert rc != 0, f"mistake {name} survived every pin: {out}"


# Mistakes in the proxy-plan planner's oracle, against test_oracle_proxy.py.
PROXY_SRC = os.path.join(ROOT, "oracle", "proxy_oracle.c")
PROXY_MUTANTS = {
    "roofline_min_not_max": ("o->load[i] = compute > memory ? compute : memory;",
                             "o->load[i] = compute < memory ? compute : memory;"),
    "traffic_without_batch": ("M += (double)jb->p[l] + (double)jb->Bg * (double)jb->a[l];",
                              "M += (double)jb->p[l] + (double)jb->a[l];"),
    "operator_bounds_rounded_up": ("o->lo[i] = (int)(((long long)i * jb->L) / O);",
                                   "o->lo[i] = (int)(((long long)i * jb->L + O - 1) / O);"),
    "bias_tie_smaller_multiset": ("(cost == st->best_cost && lex_greater(st->cur, st->best, st->s))",
                                  "(cost == st->best_cost && lex_greater(st->best, st->cur, st->s))"),
    "pairing_in_stage_order": ("double diff = (double)(1 << st->cur[st->pos[j]]) - st->D[j];",
                               "double diff = (double)(1 << st->cur[j]) - st->D[j];"),
    "lcomm_without_pipeline_term": ("*lcomm = (double)(pl->B - 1) * cmax + csum + arsum;",
                                    "*lcomm = csum + arsum;"),
    "intra_stage_tie_larger_tp": ("if (best == 0 || cost < best_cost)", "if (best == 0 || cost <= best_cost)"),
    "p2p_with_larger_dp": ("int dmin = dp < dpn ? dp : dpn;", "int dmin = dp > dpn ? dp : dpn;"),
    "proxy_tie_later_grouping": ("(b2 == bq->b2 && lcomm < bq->lcomm)", "(b2 == bq->b2 && lcomm <= bq->lcomm)"),
    "stage_allreduce_not_split_by_tp": (
        "*AR = kappa * 2.0 * (double)(dp - 1) / (double)dp * (P / (double)tp) / B_dp;",
        "*AR = kappa * 2.0 * (double)(dp - 1) / (double)dp * P / B_dp;"),
}


def _run_proxy_pins(lib):
    env = dict(os.environ, ARENA_PROXY_ORACLE_LIB=lib)
    try:
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                            "-p", "no:xdist", os.path.join(ROOT, "tests", "test_oracle_proxy.py")],
                           capture_output=True, text=True, timeout=300, env=env, cwd=ROOT)
    except subprocess.TimeoutExpired:
        return None, "timed out"
    return r.returncode, (r.stdout + r.stderr)[-2000:]


def test_unmodified_proxy_copy_passes(tmp_path):
    rc, out = _run_proxy_pins(_build(tmp_path, "proxy_control", None, PROXY_SRC))
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(PROXY_MUTANTS))
def test_planted_proxy_mistake_is_caught(tmp_path, name):
    rc, out = _run_proxy_pins(_build(tmp_path, "proxy_" + name, PROXY_MUTANTS[name], PROXY_SRC))
    assert rc != 0, f"mistake {name} survived every pin: {out}"


# Mistakes in the scheduler's oracle (Python), against test_oracle_scheduler.py.
SCHED_SRC = os.path.join(ROOT, "oracle", "scheduler_oracle.py")
SCHED_MUTANTS = {
    "launch_tie_larger_count": ("key = (-v, int(counts[c]), g)", "key = (-v, -int(counts[c]), g)"),
    "launch_needs_spare_gpu": ("if _open(v, work, ddl) and int(counts[c]) <= free[g]:",
                               "if _open(v, work, ddl) and int(counts[c]) < free[g]:"),
    "scale_down_cost_not_per_gpu": ("/ float(int(counts[c]) - int(counts[c2]))", "/ 1.0"),
    "scale_down_any_type": ("if g < 0 or g not in usable_types:", "if g < 0:"),
    "scale_up_gain_not_per_gpu": ("gain = (t2 - t) / float(dn)", "gain = (t2 - t)"),
    "priority_rule_strict": ("if int(priority[q]) <= lam:", "if int(priority[q]) < lam:"),
    "depth_off_by_one": ("if len(log) >= depth:", "if len(log) > depth:"),
    "undo_frees_instead": ("free[g] -= int(counts[c_old]) - int(counts[alloc_count[i]])",
                           "free[g] += int(counts[c_old]) - int(counts[alloc_count[i]])"),
    "deadline_strict": ("work / v <= ddl", "work / v < ddl"),
    "scale_up_to_equal_throughput": ("if t2 > t and _open(t2, work, ddl):", "if t2 >= t and _open(t2, work, ddl):"),
    "no_priority_allowance": ("lam = max((int(p) for p in priority), default=0) + 1", "lam = 0"),
    "fair_up_helps_the_best_off": ("(best is None or r0 > best[0])", "(best is None or r0 < best[0])"),
    "fair_up_without_improvement": ("if mine is not None and mine[0] < r0 and", "if mine is not None and"),
    "fair_rho_not_per_gpu": ("return work / (v * float(n)) if v > 0.0", "return work / v if v > 0.0"),
    "fair_target_tie_larger": ("if mine is None or r2 < mine[0]:", "if mine is None or r2 <= mine[0]:"),
    "fair_down_rho_before_the_step": ("cost = _rho(float(thr[i][g][c2]), int(counts[c2]), work)",
                                      "cost = _rho(float(thr[i][g][c]), int(counts[c]), work)"),
    "fair_down_throughput_cost": ("        if fair:\n            cost = _rho(", "        if not fair:\n            cost = _rho("),
    "fair_up_ignores_deadline": ("if _open(t2, work, ddl):\n                    r2", "if t2 > 0.0:\n                    r2"),
}


def _run_sched_pins(src):
    env = dict(os.environ, ARENA_SCHED_ORACLE_SRC=src)
    try:
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                            "-p", "no:xdist", os.path.join(ROOT, "tests", "test_oracle_scheduler.py")],
                           capture_output=True, text=True, timeout=300, env=env, cwd=ROOT)
    except subprocess.TimeoutExpired:
        return None, "timed out"
    return r.returncode, (r.stdout + r.stderr)[-2000:]


def _sched_copy(tmp_path, name, patch):
    src = open(SCHED_SRC).read()
    if patch is not None:
        old, new = patch
        assert src.count(old) == 1, (name, old)
        src = src.replace(old, new)
    path = tmp_path / f"sched_{name}.py"
    path.write_text(src)
    return str(path)


def test_unmodified_scheduler_copy_passes(tmp_path):
    rc, out = _run_sched_pins(_sched_copy(tmp_path, "control", None))
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(SCHED_MUTANTS))
def test_planted_scheduler_mistake_is_caught(tmp_path, name):
    rc, out = _run_sched_pins(_sched_copy(tmp_path, name, SCHED_MUTANTS[name]))
    assert rc != 0, f"mistake {name} survived every pin: {out}"


# Mistakes in the interpolated communication latency, against test_oracle_comm_tables.py.
TAB_MUTANTS = {
    # (moving to the next segment at a sample volume is no mistake: the
    # interpolant is continuous there; skipping the search is)
    "first_segment_everywhere": ("while (k < tb->K - 1 && v > tb->vol[k]) ++k;", "(void)k;"),
    "start_up_cost_when_nothing_moves": ("if (!(v > 0.0)) return 0.0;", "if (!(v >= 0.0)) return 0.0;"),
    "tp_allreduce_count_two": (
        "v += kappa * (4.0 * tab_lat(&tabs[0], 2.0 * (double)(tp - 1) / (double)tp * b * (double)jb->x[l]));",
        "v += kappa * (2.0 * tab_lat(&tabs[0], 2.0 * (double)(tp - 1) / (double)tp * b * (double)jb->x[l]));"),
    "all_to_all_on_intra_link": ("v += kappa * tab_lat(&tabs[1], b * (double)jb->a2a[l]);",
                                 "v += kappa * tab_lat(&tabs[0], b * (double)jb->a2a[l]);"),
    "p2p_one_direction": ("if (k < pp - 1) p2p = kappa * (2.0 * tab_lat(t_pp, b * (double)jb->x[hi - 1]));",
                          "if (k < pp - 1) p2p = kappa * tab_lat(t_pp, b * (double)jb->x[hi - 1]);"),
    "allreduce_volume_not_split_by_tp": (
        "if (dp > 1) AR = kappa * tab_lat(t_dp, 2.0 * (double)(dp - 1) / (double)dp * (Pk / (double)tp));",
        "if (dp > 1) AR = kappa * tab_lat(t_dp, 2.0 * (double)(dp - 1) / (double)dp * Pk);"),
    "pipeline_link_always_intra": ("const otab* t_pp = (n <= ty->gpn) ? &tabs[0] : &tabs[1];",
                                   "const otab* t_pp = &tabs[0];"),
    "partition_with_m_ignored": ("double b = (double)jb->Bg / (double)(dp * m);\n    layer_costs_tab",
                                 "double b = (double)jb->Bg / (double)dp;\n    layer_costs_tab"),
}


def _run_tab_pins(lib):
    env = dict(os.environ, ARENA_ORACLE_LIB=lib)
    try:
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                            "-p", "no:xdist", os.path.join(ROOT, "tests", "test_oracle_comm_tables.py")],
                           capture_output=True, text=True, timeout=300, env=env, cwd=ROOT)
    except subprocess.TimeoutExpired:
        return None, "timed out"
    return r.returncode, (r.stdout + r.stderr)[-2000:]


def test_unmodified_copy_passes_the_table_pins(tmp_path):
    rc, out = _run_tab_pins(_build(tmp_path, "tab_control", None))
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(TAB_MUTANTS))
def test_planted_table_mistake_is_caught(tmp_path, name):
    rc, out = _run_tab_pins(_build(tmp_path, "tab_" + name, TAB_MUTANTS[name]))
    assert rc != 0, f"mistake {name} survived every pin: {out}"


# Mistakes in the exact-T partition (the key, its suffix recursions, the
# threshold search and the cut reconstruction), against test_oracle_exact_t.py.
EXACT_T_MUTANTS = {
    "phi_without_allreduce": ("return (E->cS * sm + E->cX * x) + E->cP * pm;", "return E->cS * sm + E->cX * x;"),
    "suffix_stage_index_off_by_one": ("if (h == INFINITY || !ext_allowed(E, i, e, pp - t, tS, tP)) continue;",
                                      "if (h == INFINITY || !ext_allowed(E, i, e, pp - t + 1, tS, tP)) continue;"),
    "inner_search_stops_at_first_pair": ("                if (X == xs) break;", "                break;"),
    "last_matching_cut_not_first": ("if (E->x[e - 1] + h == H[t * L1 + i]) { c = e; break; }",
                                    "if (E->x[e - 1] + h == H[t * L1 + i]) { c = e; }"),
    "every_stage_holds_the_first_stage_memory": (
        "return fits_sums(E->M, E->segP[lo][hi], E->segA[lo][hi], k, E->pp);",
        "return fits_sums(E->M, E->segP[lo][hi], E->segA[lo][hi], 0, E->pp);"),
    "p2p_coefficient_without_b": ("*cX = kappa * 2.0 * b / B_pp;", "*cX = kappa * 2.0 / B_pp;"),
    "steady_state_m_not_m_minus_1": ("*cS = (double)(m - 1) * b;", "*cS = (double)m * b;"),
}


def _run_exact_t_pins(lib):
    env = dict(os.environ, ARENA_ORACLE_LIB=lib)
    files = [os.path.join(ROOT, "tests", "test_oracle_exact_t.py")]
    try:
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                            "-p", "no:xdist"] + files, capture_output=True, text=True, timeout=300, env=env,
                           cwd=ROOT)
    except subprocess.TimeoutExpired:
        return None, "timed out"
    return r.returncode, (r.stdout + r.stderr)[-2000:]


def test_unmodified_copy_passes_the_exact_t_pins(tmp_path):
    rc, out = _run_exact_t_pins(_build(tmp_path, "control_exact_t", None))
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(EXACT_T_MUTANTS))
def test_planted_exact_t_mistake_is_caught(tmp_path, name):
    rc, out = _run_exact_t_pins(_build(tmp_path, name, EXACT_T_MUTANTS[name]))
    assert rc != 0, f"mistake {name} survived every pin: {out}"
