"""The no-allocation estimate (arena_estimate_noalloc) against arena_estimate,
through the C ABI on the GPU.

Two calls in a row on one device, the second with a smaller workload, each
bitwise equal (times, throughputs, packed plans, cut rows, tallies) to what
arena_estimate writes for the same bindings; a workload beyond the static
scratch is refused with nothing written; the workspace cap of the allocating
entry point refuses the same way and lifts.
"""
import sys

import numpy as np
import pytest

from paper_2403_16125_amd import arena
from paper_2403_16125_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[noalloc]", *a, flush=True)
    sys.stdout.flush()


def _outputs(est):
    r = est.results()
    out = dict(t_iter=r["t_iter"].copy(), thr=r["thr"].copy(), plan=est.plan.cpu().numpy().copy())
    if est.cuts is not None:
        out["cuts"] = est.cuts.cpu().numpy().copy()
    return out


def _assert_same(a, b, what):
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), f"{what}: {k} differs"


def _both(w, rnd=0, with_cuts=True, rule=arena.PARTITION_BALANCED):
    est = arena.Estimator(w, with_cuts=with_cuts, rule=rule)
    try:
        if rnd:
            est.set_round(rnd)
        est.estimate()
        ref, cref = _outputs(est), est.counters()
        for v in (est.t_iter, est.thr, est.plan):
            v.fill_(-7)
        if est.cuts is not None:
            est.cuts.fill_(0x5A)
        est.estimate(noalloc=True)
        got, cgot = _outputs(est), est.counters()
    finally:
        est.close()
    return ref, cref, got, cgot


def test_noalloc_matches_estimate_twice_second_smaller():
    # first call: the small workload (1344 cells), second: the tiny one (32 cells)
    for name in ("small", "tiny"):
        w = wl.make(name)
        _say(f"{name}: {w.n_cells} cells, arena_estimate then arena_estimate_noalloc")
        ref, cref, got, cgot = _both(w)
        _assert_same(ref, got, name)
        assert cref == cgot, (cref, cgot)
        assert cgot["cells"] == w.n_cells


def test_noalloc_full_round_and_memory_rule():
    w = wl.full()
    _say(f"full round 3: {w.n_cells} cells without cut rows (0.7 MB of tables and 8.3 MiB of split caches "
         "in the scratch)")
    ref, cref, got, cgot = _both(w, rnd=3, with_cuts=False)
    _assert_same(ref, got, "full round 3")
    assert cref == cgot
    w = wl.make("small")
    _say("small under the memory rule, with cut rows")
    ref, cref, got, cgot = _both(w, rule=arena.PARTITION_MEMORY)
    _assert_same(ref, got, "small, memory rule")
    assert cref == cgot


def test_noalloc_refuses_beyond_scratch_and_workspace_cap():
    import torch
    w = wl.make("small")
    est = arena.Estimator(w, with_cuts=True)
    try:
        # the workspace cap of the allocating entry point: refused, nothing written
        for v in (est.t_iter, est.thr, est.plan):
            v.fill_(-7)
        est.set_workspace_limit(1024)      # the small workload needs about 2.8 KB
        with pytest.raises(arena.ArenaError) as ei:
            est.estimate()
        assert ei.value.status == arena.ARENA_ERR_OUT_OF_MEMORY
        torch.cuda.synchronize()
        assert bool((est.t_iter == -7).all()) and bool((est.plan == -7).all())
        est.set_workspace_limit(0)
        est.estimate()
        first = _outputs(est)
        # 1,000,000 jobs x 3 types: the work order and job tables need 20 MB, more
        # than the scratch holds; refused before anything is enqueued
        n = 1_000_000
        off = (np.arange(n + 1) * 4).astype(np.int32)
        fake = est.t.data_ptr()          # never read: the size check comes first
        arena.arena_bind_jobs(est.ctx, off, np.full(n, 8, np.int32), fake, fake, fake, fake, fake)
        with pytest.raises(arena.ArenaError) as ei:
            arena.arena_estimate_noalloc(est.ctx, est.t_iter, est.thr, est.plan, est.cuts,
                                         arena.CUTS_STRIDE)
        assert ei.value.status == arena.ARENA_ERR_OUT_OF_MEMORY, str(ei.value)
        torch.cuda.synchronize()
        _assert_same(first, _outputs(est), "after the refused call")
    finally:
        est.close()
