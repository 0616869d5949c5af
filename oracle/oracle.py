"""ctypes front end of the CPU oracle (arena_oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke entry and the benchmark's
CPU-baseline leg are the only callers.  Nothing here imports the HIP library
or its binding; inputs are plain numpy arrays (any object with the workload
attribute names works).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "arena_oracle.c")
_LIB = os.path.join(_HERE, "_build", "liboracle.so")

_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")

_lib = None


# gcc flags of the oracle: IEEE double, no contraction, no fast-math
CFLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra"]


def build(out: str = None, extra_flags=()) -> str:
    """Compile the oracle with gcc: IEEE double, no contraction, no fast-math.

    `extra_flags` (e.g. a sanitizer build for the tests) are appended;
    `out` defaults to the library the wrappers load."""
    out = out or _LIB
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp"
    cmd = ["gcc"] + CFLAGS + list(extra_flags) + ["-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    c_int, c_double = ctypes.c_int, ctypes.c_double
    lib.oracle_prefix.argtypes = [_f64p, c_int, _f64p]
    lib.oracle_prefix.restype = None
    lib.oracle_bottleneck_bruteforce.argtypes = [_f64p, c_int, c_int, _i32p]
    lib.oracle_bottleneck_bruteforce.restype = c_double
    lib.oracle_bottleneck_dp.argtypes = [_f64p, c_int, c_int]
    lib.oracle_bottleneck_dp.restype = c_double
    lib.oracle_canonical_cuts.argtypes = [_f64p, c_int, c_int, c_double, _i32p]
    lib.oracle_canonical_cuts.restype = None
    tables = [_i32p, _f32p, _f32p, _f32p, _f32p, _f32p, _i32p, _f32p, _f32p, _f32p, _f32p, _i32p]
    lib.oracle_bottleneck_mem.argtypes = [_f64p, _f64p, _f64p, c_int, c_int, c_int, c_double, c_int,
                                          c_double, c_int, _i32p]
    lib.oracle_bottleneck_mem.restype = c_double
    lib.oracle_exact_t.argtypes = [_f64p, _f64p, _f64p, _f64p, c_int, c_int, c_int, c_double, c_int, c_double,
                                   c_double, c_double, c_double, c_int, _i32p, _f64p]
    lib.oracle_exact_t.restype = c_double
    lib.oracle_eval_plan.argtypes = [c_int, c_int, c_int, c_double, c_int, c_int, c_int, c_int] + tables + [
        ctypes.c_void_p, ctypes.c_void_p, _f64p, c_int]
    lib.oracle_eval_plan.restype = c_int
    lib.oracle_cells.argtypes = [c_int, _i64p, c_int, c_int] + tables + [
        _i32p, _f32p, _i32p, c_int, c_double, _f64p, _i32p, _i32p, c_int, _i32p, c_int]
    lib.oracle_cells.restype = c_int
    lib.oracle_layer_costs.argtypes = [c_int, c_int, c_double, c_int, c_int] + tables + [_f64p]
    lib.oracle_layer_costs.restype = None
    lib.oracle_tab_latency.argtypes = [c_int, _f64p, _f64p, c_double]
    lib.oracle_tab_latency.restype = c_double
    lib.oracle_eval_plan_tab.argtypes = [c_int, c_int, c_int, c_double, c_int, c_int, c_int, c_int] + tables + [
        c_int, _f64p, _f64p, ctypes.c_void_p, ctypes.c_void_p, _f64p]
    lib.oracle_eval_plan_tab.restype = c_int
    lib.oracle_cells_tab.argtypes = [c_int, _i64p, c_int, c_int] + tables + [
        _i32p, _f32p, _i32p, c_int, c_double, c_int, _f64p, _f64p, _f64p, _i32p, _i32p, c_int, _i32p]
    lib.oracle_cells_tab.restype = c_int
    _lib = lib
    return lib


# ------------------------------------------------------------ partition helpers

def prefix(u) -> np.ndarray:
    u = np.ascontiguousarray(u, np.float64)
    U = np.zeros(len(u) + 1, np.float64)
    load().oracle_prefix(u, len(u), U)
    return U


def bottleneck_bruteforce(U, pp: int):
    """(W*, lexicographically smallest optimal cuts) by enumerating every cut vector."""
    U = np.ascontiguousarray(U, np.float64)
    cuts = np.zeros(max(pp - 1, 1), np.int32)
    w = load().oracle_bottleneck_bruteforce(U, len(U) - 1, pp, cuts)
    return w, [int(c) for c in cuts[:pp - 1]]


def bottleneck_dp(U, pp: int) -> float:
    U = np.ascontiguousarray(U, np.float64)
    return load().oracle_bottleneck_dp(U, len(U) - 1, pp)


def canonical_cuts(U, pp: int, W: float):
    U = np.ascontiguousarray(U, np.float64)
    cuts = np.zeros(max(pp - 1, 1), np.int32)
    load().oracle_canonical_cuts(U, len(U) - 1, pp, float(W), cuts)
    return [int(c) for c in cuts[:pp - 1]]


def bottleneck_mem(U, p, a, pp: int, m: int, b: float, tp: int, mem: float, brute: bool = False):
    """(W*_mem, cuts) of the partition whose every stage fits memory: stage k of
    pp holds 4 P/tp + min(m, pp-k) b A/tp bytes <= mem.  W = inf and cuts None
    when no split fits.  brute=True enumerates every cut vector."""
    U = np.ascontiguousarray(U, np.float64)
    p = np.ascontiguousarray(p, np.float64)
    a = np.ascontiguousarray(a, np.float64)
    cuts = np.zeros(max(pp - 1, 1), np.int32)
    w = load().oracle_bottleneck_mem(U, p, a, len(U) - 1, int(pp), int(m), float(b), int(tp), float(mem),
                                     int(bool(brute)), cuts)
    if not np.isfinite(w):
        return w, None
    return w, [int(c) for c in cuts[:pp - 1]]


def exact_t(U, p, a, x, pp: int, m: int, b: float, tp: int, mem: float, cS: float, cX: float, cP: float,
            brute: bool = False):
    """The exact-T partition of one problem: among the cut vectors whose every
    stage fits memory, the least Phi = (cS Smax + cX X) + cP Pmax (ties: least
    Smax, Pmax, X, then the lexicographically smallest cuts).  Returns
    (Phi, cuts, (Phi, Smax, Pmax, X)); Phi = inf and cuts None when no split
    fits.  brute=True enumerates every cut vector."""
    U = np.ascontiguousarray(U, np.float64)
    p = np.ascontiguousarray(p, np.float64)
    a = np.ascontiguousarray(a, np.float64)
    x = np.ascontiguousarray(x, np.float64)
    cuts = np.zeros(max(pp - 1, 1), np.int32)
    out = np.zeros(4, np.float64)
    phi = load().oracle_exact_t(U, p, a, x, len(U) - 1, int(pp), int(m), float(b), int(tp), float(mem),
                                float(cS), float(cX), float(cP), int(bool(brute)), cuts, out)
    if not np.isfinite(phi):
        return phi, None, None
    return phi, [int(c) for c in cuts[:pp - 1]], tuple(float(v) for v in out)


# ------------------------------------------------------------ workload access

def _tables(w):
    c = np.ascontiguousarray
    return (c(w.layer_offset, np.int32), c(w.t, np.float32), c(w.p, np.float32),
            c(w.a, np.float32), c(w.x, np.float32), c(w.a2a, np.float32),
            c(w.batch, np.int32), c(w.speed, np.float32), c(w.mem, np.float32),
            c(w.bw_intra, np.float32), c(w.bw_inter, np.float32),
            c(w.gpus_per_node, np.int32))


def layer_costs(w, j, g, kappa, dp, tp) -> np.ndarray:
    L = int(w.layer_offset[j + 1] - w.layer_offset[j])
    u = np.zeros(L, np.float64)
    load().oracle_layer_costs(int(j), int(g), float(kappa), int(dp), int(tp), *_tables(w), u)
    return u


def eval_plan(w, j, g, n, kappa, dp, tp, pp, m, cuts=None, rule: int = 0):
    """Price one plan.  cuts=None uses the partition of the partition rule (0:
    balanced, memory checked after; 1: balanced among the splits that fit
    memory; 2: exact-T, the least iteration time among the splits that fit).
    Returns dict(T, mem_max, s_max, feasible, cuts)."""
    out = np.zeros(4, np.float64)
    cuts_out = np.zeros(max(pp - 1, 1), np.int32)
    cin = None
    keep = None
    if cuts is not None:
        keep = np.ascontiguousarray(np.asarray(list(cuts) + [0], np.int32))
        cin = keep.ctypes.data
    rc = load().oracle_eval_plan(int(j), int(g), int(n), float(kappa), int(dp), int(tp), int(pp),
                                 int(m), *_tables(w), cin, cuts_out.ctypes.data, out, int(rule))
    if rc != 0:
        raise ValueError("oracle_eval_plan rejected the plan")
    return dict(T=out[0], mem_max=out[1], s_max=out[2], feasible=bool(out[3]),
                cuts=[int(c) for c in cuts_out[:pp - 1]])


def cells(w, cell_ids, kappa_round: int = 0, cuts_stride: int = 128, rule: int = 0):
    """Best plan of each listed cell (flat index (j*T + g)*NC + ci) under
    partition rule `rule` (see eval_plan).
    Returns dict of arrays: T (f64), thr (f64), dp, tp, pp, m (i32), cuts (i32, -1 padded),
    nplans (i32)."""
    ids = np.ascontiguousarray(np.asarray(cell_ids, np.int64))
    n = len(ids)
    res = np.zeros(2 * max(n, 1), np.float64)
    plan = np.zeros(4 * max(n, 1), np.int32)
    cuts = np.zeros(max(n, 1) * cuts_stride, np.int32)
    nplans = np.zeros(max(n, 1), np.int32)
    kap = np.ascontiguousarray(w.kappa[kappa_round], np.float32)
    rc = load().oracle_cells(n, ids, int(w.n_types), int(w.n_counts), *_tables(w),
                             np.ascontiguousarray(w.counts, np.int32), kap,
                             np.ascontiguousarray(w.m_values, np.int32), len(w.m_values),
                             float(w.tie_eps), res, plan, cuts, cuts_stride, nplans, int(rule))
    if rc != 0:
        raise ValueError("oracle_cells rejected the input")
    res = res[:2 * n].reshape(n, 2)
    plan = plan[:4 * n].reshape(n, 4)
    return dict(T=res[:, 0], thr=res[:, 1], dp=plan[:, 0], tp=plan[:, 1], pp=plan[:, 2],
                m=plan[:, 3], cuts=cuts[:n * cuts_stride].reshape(n, cuts_stride),
                nplans=nplans[:n])


# ------------------------------------------------------------ interpolated communication tables

def _tab_arrays(w, tables):
    vol = np.ascontiguousarray(tables[0], np.float64)
    lat = np.ascontiguousarray(tables[1], np.float64)
    assert vol.shape == lat.shape and vol.ndim == 3 and vol.shape[:2] == (int(w.n_types), 2)
    return vol.shape[2], vol.ravel(), lat.ravel()


def tab_latency(vol, lat, v: float) -> float:
    """Latency of v bytes in one (volume, latency) table (0 when nothing moves)."""
    vol = np.ascontiguousarray(vol, np.float64)
    lat = np.ascontiguousarray(lat, np.float64)
    return load().oracle_tab_latency(len(vol), vol, lat, float(v))


def eval_plan_tab(w, j, g, n, kappa, dp, tp, pp, m, tables, cuts=None):
    """Price one plan with communication latency from tables = (vol, lat), each
    [n_types][2 links][K].  cuts=None: the balanced partition of the plan's own
    per-microbatch costs.  Returns dict(T, mem_max, w_max, feasible, cuts)."""
    K, vol, lat = _tab_arrays(w, tables)
    out = np.zeros(4, np.float64)
    cuts_out = np.zeros(max(pp - 1, 1), np.int32)
    cin = None
    keep = None
    if cuts is not None:
        keep = np.ascontiguousarray(np.asarray(list(cuts) + [0], np.int32))
        cin = keep.ctypes.data
    rc = load().oracle_eval_plan_tab(int(j), int(g), int(n), float(kappa), int(dp), int(tp), int(pp), int(m),
                                     *_tables(w), K, vol, lat, cin, cuts_out.ctypes.data, out)
    if rc != 0:
        raise ValueError("oracle_eval_plan_tab rejected the plan")
    return dict(T=out[0], mem_max=out[1], w_max=out[2], feasible=bool(out[3]),
                cuts=[int(c) for c in cuts_out[:pp - 1]])


def cells_tab(w, cell_ids, tables, kappa_round: int = 0, cuts_stride: int = 128):
    """cells() with communication latency from tables = (vol, lat)."""
    K, vol, lat = _tab_arrays(w, tables)
    ids = np.ascontiguousarray(np.asarray(cell_ids, np.int64))
    n = len(ids)
    res = np.zeros(2 * max(n, 1), np.float64)
    plan = np.zeros(4 * max(n, 1), np.int32)
    cuts = np.zeros(max(n, 1) * cuts_stride, np.int32)
    nplans = np.zeros(max(n, 1), np.int32)
    kap = np.ascontiguousarray(w.kappa[kappa_round], np.float32)
    rc = load().oracle_cells_tab(n, ids, int(w.n_types), int(w.n_counts), *_tables(w),
                                 np.ascontiguousarray(w.counts, np.int32), kap,
                                 np.ascontiguousarray(w.m_values, np.int32), len(w.m_values),
                                 float(w.tie_eps), K, vol, lat, res, plan, cuts, cuts_stride, nplans)
    if rc != 0:
        raise ValueError("oracle_cells_tab rejected the input")
    res = res[:2 * n].reshape(n, 2)
    plan = plan[:4 * n].reshape(n, 4)
    return dict(T=res[:, 0], thr=res[:, 1], dp=plan[:, 0], tp=plan[:, 1], pp=plan[:, 2],
                m=plan[:, 3], cuts=cuts[:n * cuts_stride].reshape(n, cuts_stride),
                nplans=nplans[:n])
