"""ctypes front end of the CPU oracle of the proxy-plan planner (proxy_oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite and the benchmark's CPU-baseline leg
are the only callers.  Nothing here imports the HIP library or its binding;
inputs are numpy arrays or workload objects (workloads.Workload attribute
names).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "proxy_oracle.c")
_LIB = os.path.join(_HERE, "_build", "libproxy_oracle.so")

_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")

PLAN_WORDS = 49        # one grid: bounds[17], GPUs per stage[16], tp per stage[16]
CELL_WORDS = 52        # one cell: s, B, bounds[17], GPUs per stage[16], tp per stage[16], pad
_lib = None


# gcc flags of the oracle: IEEE double, no contraction, no fast-math
CFLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra"]


def build(out: str = None, extra_flags=()) -> str:
    """Compile with gcc: IEEE double, no contraction, no fast-math.

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
    tables = [_i32p, _f32p, _f32p, _f32p, _f32p, _f32p, _i32p, _f32p, _f32p, _f32p, _f32p, _i32p, _f32p]
    lib.proxy_oracle_normalize.argtypes = [_f64p, c_int, c_int, _i32p]
    lib.proxy_oracle_normalize.restype = c_double
    lib.proxy_oracle_loads.argtypes = [c_int, c_int, c_int] + tables + [c_double, c_int, _f64p]
    lib.proxy_oracle_loads.restype = c_int
    lib.proxy_oracle_price.argtypes = [c_int, c_int, c_int, c_double, c_int, c_int, _i32p, _i32p, _i32p] + \
        tables + [c_double, c_int, _f64p]
    lib.proxy_oracle_price.restype = c_int
    lib.proxy_oracle_grid.argtypes = [c_int, c_int, c_int, c_double, c_int, c_int] + tables + \
        [c_double, c_int, _f64p, _i32p]
    lib.proxy_oracle_grid.restype = c_int
    lib.proxy_oracle_cells.argtypes = [c_int, _i64p, c_int, c_int] + tables + \
        [_i32p, _f32p, _i32p, c_int, c_double, c_double, c_int, _f64p, _i32p]
    lib.proxy_oracle_cells.restype = c_int
    _lib = lib
    return lib


def _tables(w):
    c = lambda v, dt: np.ascontiguousarray(v, dt)
    return (c(w.layer_offset, np.int32), c(w.t, np.float32), c(w.p, np.float32), c(w.a, np.float32),
            c(w.x, np.float32), c(w.a2a, np.float32), c(w.batch, np.int32), c(w.speed, np.float32),
            c(w.mem, np.float32), c(w.bw_intra, np.float32), c(w.bw_inter, np.float32),
            c(w.gpus_per_node, np.int32), c(w.hbm_bw(), np.float32))


def normalize(D, n: int):
    """(squared computation bias, power-of-two GPUs per stage) or (None, None)."""
    D = np.ascontiguousarray(D, np.float64)
    m = np.zeros(max(1, len(D)), np.int32)
    b2 = load().proxy_oracle_normalize(D, len(D), int(n), m)
    if b2 < 0:
        return None, None
    return b2, m[: len(D)].copy()


def loads(w, j: int, g: int, n: int, f_ref: float, n_ops: int = 16):
    out = np.zeros(2 * 16, np.float64)
    O = load().proxy_oracle_loads(j, g, n, *_tables(w), float(f_ref), int(n_ops), out)
    if O < 0:
        raise ValueError("bad job")
    return out[:O].copy(), out[O:2 * O].copy()


def price(w, j: int, g: int, n: int, kappa: float, bounds, Dn, tp, B: int, f_ref: float,
          n_ops: int = 16):
    """(T, feasible, l_comm) of a plan with stage boundaries at operators."""
    bounds = np.ascontiguousarray(bounds, np.int32)
    s = len(bounds) - 1
    out = np.zeros(3, np.float64)
    rc = load().proxy_oracle_price(j, g, n, float(kappa), s, int(B), bounds,
                                   np.ascontiguousarray(Dn, np.int32), np.ascontiguousarray(tp, np.int32),
                                   *_tables(w), float(f_ref), int(n_ops), out)
    if rc:
        raise ValueError("bad plan")
    return float(out[0]), bool(out[1]), float(out[2])


def grid(w, j: int, g: int, n: int, kappa: float, s: int, B: int, f_ref: float, n_ops: int = 16):
    """The proxy plan of grid (s, B): dict ok, b2, lcomm, T, bounds, Dn, tp."""
    out = np.zeros(4, np.float64)
    plan = np.zeros(PLAN_WORDS, np.int32)
    rc = load().proxy_oracle_grid(j, g, n, float(kappa), s, int(B), *_tables(w), float(f_ref),
                                  int(n_ops), out, plan)
    if rc:
        raise ValueError("bad grid")
    return dict(ok=bool(out[0]), b2=float(out[1]), lcomm=float(out[2]), T=float(out[3]),
                bounds=plan[: s + 1].copy(), Dn=plan[17:17 + s].copy(), tp=plan[33:33 + s].copy())


def cells(w, ids, kappa_round: int = 0, f_ref: float = 1e14, n_ops: int = 16) -> dict:
    """The proxy-estimated best plan of each listed cell id ((j T + g) NC + c)."""
    ids = np.ascontiguousarray(ids, np.int64)
    out = np.zeros((len(ids), 4), np.float64)
    plan = np.zeros((len(ids), CELL_WORDS), np.int32)
    kap = np.ascontiguousarray(np.asarray(w.kappa)[kappa_round], np.float32)
    rc = load().proxy_oracle_cells(len(ids), ids, w.n_types, w.n_counts, *_tables(w),
                                   np.ascontiguousarray(w.counts, np.int32), kap,
                                   np.ascontiguousarray(w.m_values, np.int32), len(w.m_values),
                                   float(w.tie_eps), float(f_ref), int(n_ops), out, plan)
    if rc:
        raise ValueError("bad cell")
    return dict(T=out[:, 0], b2=out[:, 1], lcomm=out[:, 2], thr=out[:, 3], s=plan[:, 0], B=plan[:, 1],
                bounds=plan[:, 2:19], Dn=plan[:, 19:35], tp=plan[:, 35:51])
