"""The memory-constrained partition's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of the oracle's C source (an in-flight
count off by one, the tensor degree dropped from the activations, a strict
memory limit, stages counted from the wrong end, the microbatch size missing
its m, a cut search that allows empty stages or completes with one stage too
few, a sum where the recursion takes a maximum), builds it with gcc into a
temporary library, and runs the pins of test_oracle_memory_partition.py
against it in a child process: some pin must fail (an assertion, or a crash
or time-out of the broken copy).  The unmodified copy, built the same way,
must pass them all.
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
    "microbatch_size_without_m": ("M.b = (double)jb->Bg / (double)(dp * m);",
                                  "M.b = (double)jb->Bg / (double)dp;"),
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


def _build(tmp_path, name, patch):
    src = open(SRC).read()
    if patch is not None:
        old, new = patch
        assert src.count(old) == 1, (name, old)
        src = src.replace(old, new)
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
    rc, out = _run_pins(_build(tmp_path, "control", None))
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    rc, out = _run_pins(_build(tmp_path, name, MUTANTS[name]))
    assert rc != 0, f"mistake {name} survived every pin: {out}"
