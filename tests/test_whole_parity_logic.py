"""CPU check of the comparison in tests/whole_workload_parity.py: GPU-format
outputs built from the oracle's own results settle as exact, and a planted
difference in the plan, the cuts or the time is left to the per-cell
comparison, which reports it."""
import numpy as np

from compare import compare, select
from paper_2403_16125_amd import workloads as wl
import whole_workload_parity as wp


def _as_gpu(ref):
    n = len(ref["T"])
    feas = np.isfinite(ref["T"])
    cuts = np.full((n, 128), 0xFF, np.uint8)
    for s in np.nonzero(feas)[0]:
        pp = int(ref["pp"][s])
        cuts[s, :pp - 1] = ref["cuts"][s, :pp - 1]
    z = lambda k: np.where(feas, ref[k], 0).astype(np.int32)
    return dict(t_iter=np.where(feas, ref["T"], np.inf).astype(np.float32),
                thr=np.where(feas, ref["thr"], 0.0).astype(np.float32),
                dp=z("dp"), tp=z("tp"), pp=z("pp"), m=z("m"), feasible=feas, cuts=cuts)


def test_settle_and_planted_differences(oracle):
    w = wl.make("small")
    ids = np.arange(w.n_cells)
    ref = oracle.cells(w, ids)
    gpu = _as_gpu(ref)
    ok, relT = wp.settle(gpu, ref, 0, w.n_cells)
    assert ok.all() and relT.max() < 1e-6
    feas = np.nonzero(np.isfinite(ref["T"]) & (ref["pp"] > 1))[0]
    a, b, c = (int(v) for v in feas[:3])
    gpu["m"][a] = 1 if gpu["m"][a] != 1 else 2              # another plan
    gpu["cuts"][b, 0] = (int(gpu["cuts"][b, 0]) + 1) % 100  # other cuts
    gpu["t_iter"][c] *= np.float32(1.001)                   # another time
    ok, _ = wp.settle(gpu, ref, 0, w.n_cells)
    rest = np.nonzero(~ok)[0]
    assert sorted(rest.tolist()) == sorted([a, b, c])
    rep = compare(w, select(gpu, rest), rest, oracle, ref={k: v[rest] for k, v in ref.items()})
    assert len(rep["mismatch"]) == 3 and rep["exact"] == 0


def test_settle_without_cut_rows(oracle):
    """The timed launch writes no cut rows: plans, times and throughputs are
    still settled, and a planted difference in the plan or the time is left
    to the per-cell comparison."""
    w = wl.make("small")
    ids = np.arange(w.n_cells)
    ref = oracle.cells(w, ids)
    gpu = _as_gpu(ref)
    del gpu["cuts"]
    ok, _ = wp.settle(gpu, ref, 0, w.n_cells)
    assert ok.all()
    feas = np.nonzero(np.isfinite(ref["T"]) & (ref["pp"] > 1))[0]
    a, c = int(feas[0]), int(feas[1])
    gpu["pp"][a] = 1 if gpu["pp"][a] != 1 else 2            # another plan
    gpu["t_iter"][c] *= np.float32(1.001)                   # another time
    ok, _ = wp.settle(gpu, ref, 0, w.n_cells)
    assert sorted(np.nonzero(~ok)[0].tolist()) == sorted([a, c])
