"""Host-side checks of the benchmark driver and the work counts (no GPU)."""
import math
import os
import subprocess
import sys

import numpy as np

from paper_2403_16125_amd import workcount
from paper_2403_16125_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    for extra in (["--gpus", "2"], ["--gpus", "8", "--schedule"], ["--gpus", "4", "--proxy"]):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + extra,
                           capture_output=True, text=True, timeout=120)
        assert r.returncode == 2
        assert "one GPU" in r.stderr and r.stdout == ""


def _brute_pow2_splits(n, s):
    # ordered vectors of s powers of two summing to n, counted as multisets
    pw = [1 << e for e in range(n.bit_length())]
    seen = set()

    def rec(k, left, maxp, cur):
        if k == s:
            if left == 0:
                seen.add(tuple(cur))
            return
        for p in pw:
            if p <= maxp and p <= left:
                rec(k + 1, left - p, p, cur + [p])

    rec(0, n, n, [])
    return len(seen)


def test_power_of_two_split_counts():
    for n in (1, 2, 3, 6, 8, 12, 16, 24, 40):
        top = 1 << (n.bit_length() - 1)
        for s in range(1, 9):
            assert workcount._pow2_splits(n, s, top) == _brute_pow2_splits(n, s)


def test_proxy_work_closed_forms():
    # one operator, one GPU: one grid of one grouping with one multiset
    assert workcount._proxy_cell_ops(1, 1, 3) == 3 * 1 * 1 + 8 * 1 * 3
    # O operators, n = 2: s = 1 has the split {2}, s = 2 the split {1, 1}
    O = 5
    want = math.comb(O - 1, 0) * (3 * 1 * 1 + 8 * 1 * 2) + math.comb(O - 1, 1) * (3 * 2 * 1 + 8 * 2 * 2)
    assert workcount._proxy_cell_ops(2, O, 2) == want
    # the launch total is the per-cell sum over every job, type and count
    w = wl.make("tiny")
    per_job = sum(workcount._proxy_cell_ops(int(n), 12, len(w.m_values)) for n in w.counts)
    assert workcount.proxy_ops(w) == per_job * w.n_types * w.n_jobs
    assert workcount.proxy_ops(w, n_ops=4) < workcount.proxy_ops(w)
    assert np.isfinite(workcount.proxy_ops(wl.make("small")))
