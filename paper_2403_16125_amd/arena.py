"""Python binding of libarena.so: the C ABI of include/arena.h under the same
names, plus a small `Estimator` that keeps a workload's tables resident in
device memory and a `Scheduler` that runs scheduling steps over a throughput
matrix.

This module only marshals arguments.  Every step of the estimate runs in the
HIP library; torch is used for device allocations and the current stream.
If the library is not built this module raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_build", "libarena.so")

ARENA_OK = 0
ARENA_ERR_INVALID_ARG = 1
ARENA_ERR_OUT_OF_MEMORY = 2
ARENA_ERR_DEVICE = 3
ARENA_ERR_NOT_READY = 4
ARENA_ERR_UNSUPPORTED = 5

MAX_LAYERS = 128
CUTS_STRIDE = MAX_LAYERS  # bytes of cut row per cell used by this binding

EXPORTED = (
    "arena_create", "arena_destroy", "arena_last_error", "arena_status_string",
    "arena_bind_jobs", "arena_bind_grids", "arena_set_kappa", "arena_set_plan_space",
    "arena_space_size_get", "arena_estimate", "arena_get_counters", "arena_set_bound_pruning",
    "arena_schedule", "arena_proxy_estimate", "arena_set_partition_rule", "arena_set_comm_tables",
    "arena_set_workspace_limit", "arena_estimate_noalloc",
)

NOALLOC_SCRATCH_BYTES = 16 << 20

PARTITION_BALANCED = 0
PARTITION_MEMORY = 1
PARTITION_EXACT_T = 2
EXACT_T_MAX_LAYERS = 96
SCHED_THROUGHPUT = 0
SCHED_FAIRNESS = 1
_OBJECTIVES = {"throughput": SCHED_THROUGHPUT, "fairness": SCHED_FAIRNESS}

MAX_PROXY_OPS = 16

MAX_SCHED_JOBS = 65536
MAX_SCHED_DEPTH = 256


class ArenaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status
        self.message = message


class JobsDesc(ctypes.Structure):
    _fields_ = [("n_jobs", ctypes.c_int32), ("n_layers_total", ctypes.c_int32),
                ("layer_offset", ctypes.c_void_p), ("batch", ctypes.c_void_p),
                ("t", ctypes.c_void_p), ("p", ctypes.c_void_p), ("a", ctypes.c_void_p),
                ("x", ctypes.c_void_p), ("a2a", ctypes.c_void_p)]


class GridsDesc(ctypes.Structure):
    _fields_ = [("n_types", ctypes.c_int32), ("speed", ctypes.c_void_p),
                ("mem_bytes", ctypes.c_void_p), ("bw_intra", ctypes.c_void_p),
                ("bw_inter", ctypes.c_void_p), ("gpus_per_node", ctypes.c_void_p),
                ("n_counts", ctypes.c_int32), ("counts", ctypes.c_void_p)]


class Counters(ctypes.Structure):
    _fields_ = [("cells", ctypes.c_int64), ("plans", ctypes.c_int64),
                ("problems", ctypes.c_int64), ("dp_entries", ctypes.c_int64),
                ("infeasible_cells", ctypes.c_int64), ("plans_skipped", ctypes.c_int64),
                ("alg_ops", ctypes.c_int64), ("mem_partitions", ctypes.c_int64)]


class ProxyDesc(ctypes.Structure):
    _fields_ = [("hbm_bw", ctypes.c_void_p), ("f_ref", ctypes.c_double), ("n_ops", ctypes.c_int32)]


class SchedDesc(ctypes.Structure):
    _fields_ = [("n_jobs", ctypes.c_int32), ("n_types", ctypes.c_int32), ("n_counts", ctypes.c_int32),
                ("thr", ctypes.c_void_p), ("counts", ctypes.c_void_p), ("capacity", ctypes.c_void_p),
                ("alloc_type", ctypes.c_void_p), ("alloc_count", ctypes.c_void_p),
                ("queue", ctypes.c_void_p), ("priority", ctypes.c_void_p),
                ("n_queue", ctypes.c_int32), ("depth", ctypes.c_int32),
                ("launched", ctypes.c_void_p), ("result", ctypes.c_void_p),
                ("batch", ctypes.c_void_p), ("iters", ctypes.c_void_p), ("deadline", ctypes.c_void_p),
                ("objective", ctypes.c_int32)]


class SpaceSize(ctypes.Structure):
    _fields_ = [("cells", ctypes.c_int64), ("plans", ctypes.c_int64),
                ("max_plans_per_cell", ctypes.c_int32), ("max_layers", ctypes.c_int32)]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load():
    """Load libarena.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ArenaError(ARENA_ERR_NOT_READY,
                         f"{_LIB_PATH} is missing: build it with paper_2403_16125_amd.build")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, st = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int
    lib.arena_create.argtypes = [ctypes.c_int, ctypes.POINTER(vp)]
    lib.arena_create.restype = st
    lib.arena_destroy.argtypes = [vp]
    lib.arena_destroy.restype = None
    lib.arena_last_error.argtypes = [vp]
    lib.arena_last_error.restype = ctypes.c_char_p
    lib.arena_status_string.argtypes = [st]
    lib.arena_status_string.restype = ctypes.c_char_p
    lib.arena_bind_jobs.argtypes = [vp, ctypes.POINTER(JobsDesc)]
    lib.arena_bind_jobs.restype = st
    lib.arena_bind_grids.argtypes = [vp, ctypes.POINTER(GridsDesc)]
    lib.arena_bind_grids.restype = st
    lib.arena_set_kappa.argtypes = [vp, vp, i32]
    lib.arena_set_kappa.restype = st
    lib.arena_set_plan_space.argtypes = [vp, vp, i32, ctypes.c_double]
    lib.arena_set_plan_space.restype = st
    lib.arena_set_bound_pruning.argtypes = [vp, i32]
    lib.arena_set_bound_pruning.restype = st
    lib.arena_set_partition_rule.argtypes = [vp, i32]
    lib.arena_set_partition_rule.restype = st
    lib.arena_set_comm_tables.argtypes = [vp, i32, vp, vp]
    lib.arena_set_comm_tables.restype = st
    lib.arena_space_size_get.argtypes = [vp, ctypes.POINTER(SpaceSize)]
    lib.arena_space_size_get.restype = st
    lib.arena_estimate.argtypes = [vp, vp, vp, vp, vp, i32, vp]
    lib.arena_estimate.restype = st
    lib.arena_estimate_noalloc.argtypes = [vp, vp, vp, vp, vp, i32, vp]
    lib.arena_estimate_noalloc.restype = st
    lib.arena_set_workspace_limit.argtypes = [vp, ctypes.c_int64]
    lib.arena_set_workspace_limit.restype = st
    lib.arena_get_counters.argtypes = [vp, ctypes.POINTER(Counters)]
    lib.arena_get_counters.restype = st
    lib.arena_proxy_estimate.argtypes = [vp, ctypes.POINTER(ProxyDesc), vp, vp, vp, vp]
    lib.arena_proxy_estimate.restype = st
    lib.arena_schedule.argtypes = [vp, ctypes.POINTER(SchedDesc), vp]
    lib.arena_schedule.restype = st
    _lib = lib
    return lib


def _status_name(s: int) -> str:
    names = {0: "ARENA_OK", 1: "ARENA_ERR_INVALID_ARG", 2: "ARENA_ERR_OUT_OF_MEMORY",
             3: "ARENA_ERR_DEVICE", 4: "ARENA_ERR_NOT_READY", 5: "ARENA_ERR_UNSUPPORTED"}
    return names.get(int(s), f"status {s}")


def _check(ctx, status: int):
    if status != ARENA_OK:
        msg = load().arena_last_error(ctx)
        raise ArenaError(status, msg.decode() if msg else "")


def _ptr(a) -> int:
    """Address of a numpy array or torch tensor (0 for None)."""
    if a is None:
        return 0
    if isinstance(a, (int, np.integer)):
        return int(a)
    if isinstance(a, np.ndarray):
        return a.ctypes.data
    return int(a.data_ptr())


# ---------------------------------------------------------------- raw C ABI

def arena_create(device: int = 0):
    h = ctypes.c_void_p()
    s = load().arena_create(int(device), ctypes.byref(h))
    if s != ARENA_OK:
        raise ArenaError(s, "arena_create failed")
    return h


def arena_destroy(ctx) -> None:
    load().arena_destroy(ctx)


def arena_last_error(ctx) -> str:
    m = load().arena_last_error(ctx)
    return m.decode() if m else ""


def arena_status_string(status: int) -> str:
    return load().arena_status_string(int(status)).decode()


def arena_bind_jobs(ctx, layer_offset, batch, t, p, a, x, a2a, n_layers_total=None):
    """layer_offset, batch: host int32 arrays; t..a2a: device float32 tensors (or pointers)."""
    off = np.ascontiguousarray(layer_offset, np.int32)
    bat = np.ascontiguousarray(batch, np.int32)
    d = JobsDesc(n_jobs=len(bat), n_layers_total=int(off[-1] if n_layers_total is None else n_layers_total),
                 layer_offset=_ptr(off), batch=_ptr(bat), t=_ptr(t), p=_ptr(p), a=_ptr(a),
                 x=_ptr(x), a2a=_ptr(a2a))
    _check(ctx, load().arena_bind_jobs(ctx, ctypes.byref(d)))


def arena_bind_grids(ctx, speed, mem_bytes, bw_intra, bw_inter, gpus_per_node, counts):
    f = lambda v: np.ascontiguousarray(v, np.float32)
    arrs = [f(speed), f(mem_bytes), f(bw_intra), f(bw_inter),
            np.ascontiguousarray(gpus_per_node, np.int32), np.ascontiguousarray(counts, np.int32)]
    d = GridsDesc(n_types=len(arrs[0]), speed=_ptr(arrs[0]), mem_bytes=_ptr(arrs[1]),
                  bw_intra=_ptr(arrs[2]), bw_inter=_ptr(arrs[3]), gpus_per_node=_ptr(arrs[4]),
                  n_counts=len(arrs[5]), counts=_ptr(arrs[5]))
    _check(ctx, load().arena_bind_grids(ctx, ctypes.byref(d)))


def arena_set_kappa(ctx, kappa) -> None:
    k = np.ascontiguousarray(kappa, np.float32).ravel()
    _check(ctx, load().arena_set_kappa(ctx, _ptr(k), len(k)))


def arena_set_plan_space(ctx, m_values, tie_eps: float) -> None:
    m = np.ascontiguousarray(m_values, np.int32)
    _check(ctx, load().arena_set_plan_space(ctx, _ptr(m), len(m), float(tie_eps)))


def arena_set_bound_pruning(ctx, enabled: bool) -> None:
    _check(ctx, load().arena_set_bound_pruning(ctx, 1 if enabled else 0))


def arena_set_partition_rule(ctx, rule: int) -> None:
    _check(ctx, load().arena_set_partition_rule(ctx, int(rule)))


def arena_set_comm_tables(ctx, volumes=None, latencies=None) -> None:
    """volumes, latencies: float64 [n_types][2][K] host arrays, or None to return
    to volume / bandwidth."""
    if volumes is None:
        _check(ctx, load().arena_set_comm_tables(ctx, 0, None, None))
        return
    v = np.ascontiguousarray(volumes, np.float64)
    lt = np.ascontiguousarray(latencies, np.float64)
    if v.shape != lt.shape or v.ndim != 3 or v.shape[1] != 2:
        raise ValueError("comm tables: volumes and latencies must both be [n_types][2][K]")
    _check(ctx, load().arena_set_comm_tables(ctx, int(v.shape[2]), v.ctypes.data, lt.ctypes.data))


def arena_space_size_get(ctx) -> dict:
    s = SpaceSize()
    _check(ctx, load().arena_space_size_get(ctx, ctypes.byref(s)))
    return dict(cells=s.cells, plans=s.plans, max_plans_per_cell=s.max_plans_per_cell,
                max_layers=s.max_layers)


def arena_estimate(ctx, t_iter, thr, plan, cuts=None, cuts_stride: int = 0, stream=None) -> None:
    """Outputs are device tensors (or pointers); stream is a HIP stream handle or None."""
    sp = 0 if stream is None else int(stream)
    _check(ctx, load().arena_estimate(ctx, _ptr(t_iter), _ptr(thr), _ptr(plan), _ptr(cuts),
                                      int(cuts_stride), sp))


def arena_estimate_noalloc(ctx, t_iter, thr, plan, cuts=None, cuts_stride: int = 0, stream=None) -> None:
    """arena_estimate with the library's tables in its static device scratch
    (no device allocation); arguments as arena_estimate."""
    sp = 0 if stream is None else int(stream)
    _check(ctx, load().arena_estimate_noalloc(ctx, _ptr(t_iter), _ptr(thr), _ptr(plan), _ptr(cuts),
                                              int(cuts_stride), sp))


def arena_set_workspace_limit(ctx, nbytes: int) -> None:
    _check(ctx, load().arena_set_workspace_limit(ctx, int(nbytes)))


def arena_get_counters(ctx) -> dict:
    c = Counters()
    _check(ctx, load().arena_get_counters(ctx, ctypes.byref(c)))
    return dict(cells=c.cells, plans=c.plans, problems=c.problems, dp_entries=c.dp_entries,
                infeasible_cells=c.infeasible_cells, plans_skipped=c.plans_skipped, alg_ops=c.alg_ops,
                mem_partitions=c.mem_partitions)


def arena_proxy_estimate(ctx, hbm_bw, f_ref: float, n_ops: int, t_iter, thr, plan, stream=None) -> None:
    """hbm_bw: host f32 [n_types]; outputs are device tensors (or pointers)."""
    hbm = np.ascontiguousarray(hbm_bw, np.float32)
    d = ProxyDesc(_ptr(hbm), float(f_ref), int(n_ops))
    sp = 0 if stream is None else int(stream)
    _check(ctx, load().arena_proxy_estimate(ctx, ctypes.byref(d), _ptr(t_iter), _ptr(thr), _ptr(plan), sp))


def unpack_proxy_plan(words):
    """[C, 3] uint64 plan words -> dict of s, B, feasible, stage-start mask,
    GPUs and tensor degree per stage ([C, 16], 0 past the last stage)."""
    w = np.asarray(words, np.uint64).reshape(-1, 3)
    w0 = w[:, 0]
    s = ((w0 >> np.uint64(16)) & np.uint64(31)).astype(np.int32)
    out = dict(s=s, B=((w0 >> np.uint64(24)) & np.uint64(127)).astype(np.int32),
               feasible=((w0 >> np.uint64(31)) & np.uint64(1)).astype(bool),
               starts=(w0 & np.uint64(0x7FFF)).astype(np.int64))
    k = np.arange(16, dtype=np.uint64)
    dexp = ((w[:, 1:2] >> (np.uint64(4) * k)) & np.uint64(15)).astype(np.int64)
    texp = ((w[:, 2:3] >> (np.uint64(4) * k)) & np.uint64(15)).astype(np.int64)
    live = np.arange(16)[None, :] < s[:, None]
    out["Dn"] = np.where(live, 1 << dexp, 0).astype(np.int32)
    out["tp"] = np.where(live, 1 << texp, 0).astype(np.int32)
    return out


def arena_schedule(ctx, n_jobs, n_types, n_counts, thr, counts, capacity, alloc_type, alloc_count,
                   queue, priority, n_queue, depth, launched, result, stream=None,
                   batch=None, iters=None, deadline=None, objective=0) -> None:
    """thr, alloc_type, alloc_count, queue, priority, launched, result and the
    optional batch / iters / deadline arrays are device tensors (or pointers);
    counts and capacity are host int32 arrays.  objective: SCHED_THROUGHPUT or
    SCHED_FAIRNESS."""
    counts = np.ascontiguousarray(counts, np.int32)
    capacity = np.ascontiguousarray(capacity, np.int32)
    d = SchedDesc(int(n_jobs), int(n_types), int(n_counts), _ptr(thr), _ptr(counts), _ptr(capacity),
                  _ptr(alloc_type), _ptr(alloc_count), _ptr(queue), _ptr(priority), int(n_queue),
                  int(depth), _ptr(launched), _ptr(result), _ptr(batch), _ptr(iters), _ptr(deadline),
                  int(objective))
    sp = 0 if stream is None else int(stream)
    _check(ctx, load().arena_schedule(ctx, ctypes.byref(d), sp))


# ---------------------------------------------------------------- convenience

def unpack_plan(words):
    w = np.asarray(words).astype(np.uint32)
    return dict(dp=(w & 0x7FF).astype(np.int32), tp=((w >> 11) & 0x1F).astype(np.int32),
                pp=((w >> 16) & 0xFF).astype(np.int32), m=((w >> 24) & 0x7F).astype(np.int32),
                feasible=((w >> 31) & 1).astype(bool))


class Estimator:
    """Binds a workload's tables (resident in device memory) and runs rounds.

    `workload` is any object with the attributes of workloads.Workload."""

    def __init__(self, workload, device: int = 0, with_cuts: bool = False, prune: bool = True,
                 rule: int = PARTITION_BALANCED, comm_tables=None):
        import torch
        self.torch = torch
        self.w = workload
        self.dev = torch.device("cuda", device)
        load()
        self.ctx = arena_create(device)
        self._alive = True
        try:
            tens = lambda v: torch.as_tensor(np.ascontiguousarray(v, np.float32)).to(self.dev)
            self.t, self.p, self.a, self.x, self.a2a = (tens(workload.t), tens(workload.p),
                                                        tens(workload.a), tens(workload.x),
                                                        tens(workload.a2a))
            arena_bind_jobs(self.ctx, workload.layer_offset, workload.batch,
                            self.t, self.p, self.a, self.x, self.a2a)
            arena_bind_grids(self.ctx, workload.speed, workload.mem, workload.bw_intra,
                             workload.bw_inter, workload.gpus_per_node, workload.counts)
            arena_set_plan_space(self.ctx, workload.m_values, workload.tie_eps)
            arena_set_kappa(self.ctx, workload.kappa[0])
            arena_set_bound_pruning(self.ctx, prune)
            arena_set_partition_rule(self.ctx, rule)
            if comm_tables is not None:
                arena_set_comm_tables(self.ctx, *comm_tables)
            C = workload.n_cells
            self.n_cells = C
            self.t_iter = torch.empty(C, dtype=torch.float32, device=self.dev)
            self.thr = torch.empty(C, dtype=torch.float32, device=self.dev)
            self.plan = torch.empty(C, dtype=torch.int32, device=self.dev)
            self.cuts = (torch.empty(C * CUTS_STRIDE, dtype=torch.uint8, device=self.dev)
                         if with_cuts else None)
        except Exception:
            self.close()
            raise

    def set_round(self, r: int) -> None:
        arena_set_kappa(self.ctx, self.w.kappa[r])

    def set_kappa(self, kappa) -> None:
        arena_set_kappa(self.ctx, kappa)

    def set_partition_rule(self, rule: int) -> None:
        arena_set_partition_rule(self.ctx, rule)

    def set_comm_tables(self, tables=None) -> None:
        """tables = (volumes, latencies), each [n_types][2][K]; None: volume / bandwidth."""
        if tables is None:
            arena_set_comm_tables(self.ctx)
        else:
            arena_set_comm_tables(self.ctx, *tables)

    def estimate(self, stream=None, noalloc: bool = False) -> None:
        """Estimate every cell into the estimator's outputs; noalloc=True takes
        the entry point that allocates nothing (its tables in the library's
        static device scratch)."""
        s = self.torch.cuda.current_stream(self.dev) if stream is None else stream
        fn = arena_estimate_noalloc if noalloc else arena_estimate
        fn(self.ctx, self.t_iter, self.thr, self.plan, self.cuts,
           CUTS_STRIDE if self.cuts is not None else 0, s.cuda_stream)

    def set_workspace_limit(self, nbytes: int) -> None:
        arena_set_workspace_limit(self.ctx, nbytes)

    def proxy_estimate(self, f_ref: float = 1e14, n_ops: int = 16, hbm_bw=None, stream=None) -> None:
        """The proxy-plan planner over the same cells (outputs kept beside the
        estimate's)."""
        torch = self.torch
        if getattr(self, "p_t_iter", None) is None:
            C = self.n_cells
            self.p_t_iter = torch.empty(C, dtype=torch.float32, device=self.dev)
            self.p_thr = torch.empty(C, dtype=torch.float32, device=self.dev)
            self.p_plan = torch.empty(C * 3, dtype=torch.int64, device=self.dev)
        hbm = self.w.hbm_bw() if hbm_bw is None else hbm_bw
        s = torch.cuda.current_stream(self.dev) if stream is None else stream
        arena_proxy_estimate(self.ctx, hbm, f_ref, n_ops, self.p_t_iter, self.p_thr, self.p_plan,
                             s.cuda_stream)

    def proxy_results(self, ids=None) -> dict:
        torch = self.torch
        torch.cuda.synchronize(self.dev)
        if ids is None:
            sel = lambda v: v
        else:
            idx = torch.as_tensor(np.asarray(ids, np.int64), device=self.dev)
            sel = lambda v: v.index_select(0, idx)
        words = sel(self.p_plan.view(self.n_cells, 3)).cpu().numpy().view(np.uint64)
        out = dict(t_iter=sel(self.p_t_iter).cpu().numpy(), thr=sel(self.p_thr).cpu().numpy(),
                   words=words)
        out.update(unpack_proxy_plan(words))
        return out

    def space_size(self) -> dict:
        return arena_space_size_get(self.ctx)

    def counters(self) -> dict:
        return arena_get_counters(self.ctx)

    def results(self, ids=None) -> dict:
        """Synchronise and copy the last estimate (all cells, or the listed
        cells gathered on the device first) to host numpy arrays."""
        torch = self.torch
        torch.cuda.synchronize(self.dev)
        if ids is None:
            sel = lambda v: v
        else:
            idx = torch.as_tensor(np.asarray(ids, np.int64), device=self.dev)
            sel = lambda v: v.index_select(0, idx)
        out = dict(t_iter=sel(self.t_iter).cpu().numpy(), thr=sel(self.thr).cpu().numpy(),
                   plan=sel(self.plan).cpu().numpy().view(np.uint32))
        out.update(unpack_plan(out["plan"]))
        if self.cuts is not None:
            rows = sel(self.cuts.view(self.n_cells, CUTS_STRIDE))
            out["cuts"] = rows.cpu().numpy()
        return out

    def close(self) -> None:
        if getattr(self, "_alive", False):
            self.torch.cuda.synchronize(self.dev)
            arena_destroy(self.ctx)
            self._alive = False

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Scheduler:
    """Runs scheduling steps (arena_schedule) over a throughput matrix held in
    device memory: `thr` is a float32 [J, T, NC] array or device tensor (the
    thr output of an estimate, viewed as [J, T, NC], serves directly)."""

    def __init__(self, thr, counts, capacity, device: int = 0, batch=None, iters=None, deadline=None,
                 objective: str = "throughput"):
        import torch
        self.torch = torch
        self.dev = torch.device("cuda", device)
        load()
        self.ctx = arena_create(device)
        self._alive = True
        try:
            if isinstance(thr, torch.Tensor):
                self.thr = thr.to(self.dev, torch.float32).contiguous()
            else:
                self.thr = torch.as_tensor(np.ascontiguousarray(thr, np.float32)).to(self.dev)
            if self.thr.dim() != 3:
                raise ValueError("thr must be [jobs, types, counts]")
            self.n_jobs, self.n_types, self.n_counts = (int(v) for v in self.thr.shape)
            self.counts = np.ascontiguousarray(counts, np.int32)
            self.capacity = np.ascontiguousarray(capacity, np.int32)
            if self.counts.shape != (self.n_counts,) or self.capacity.shape != (self.n_types,):
                raise ValueError("counts / capacity do not match thr")
            i32 = dict(dtype=torch.int32, device=self.dev)
            self.alloc_type = torch.empty(self.n_jobs, **i32)
            self.alloc_count = torch.empty(self.n_jobs, **i32)
            self.queue = torch.empty(max(1, self.n_jobs), **i32)
            self.priority = torch.empty(max(1, self.n_jobs), **i32)
            self.launched = torch.empty(max(1, self.n_jobs), **i32)
            self.result = torch.empty(8, **i32)
            self.n_queue = 0
            self.set_objective(objective)
            self.batch = self.iters = self.deadline = None
            if batch is not None or iters is not None or deadline is not None:
                self.set_deadlines(batch, iters, deadline)
        except Exception:
            self.close()
            raise

    def set_objective(self, objective: str) -> None:
        """"throughput" (Eq. 5) or "fairness" (Eq. 7; needs batch and iters)."""
        if objective not in _OBJECTIVES:
            raise ValueError(f"objective must be one of {sorted(_OBJECTIVES)}")
        self.objective = _OBJECTIVES[objective]

    def set_deadlines(self, batch, iters, deadline) -> None:
        """Per-job batch, remaining iterations and deadline (Eq. 6), or all
        None; deadline alone may be None (the fairness objective's work)."""
        torch = self.torch
        if batch is None and iters is None and deadline is None:
            self.batch = self.iters = self.deadline = None
            return
        self.batch = torch.as_tensor(np.ascontiguousarray(batch, np.int32)).to(self.dev)
        self.iters = torch.as_tensor(np.ascontiguousarray(iters, np.float32)).to(self.dev)
        self.deadline = (None if deadline is None else
                         torch.as_tensor(np.ascontiguousarray(deadline, np.float32)).to(self.dev))
        torch.cuda.synchronize(self.dev)

    def load_state(self, alloc_type, alloc_count, queue, priority) -> None:
        """Copy a cluster state (allocation and queue) to the device (synchronously)."""
        torch = self.torch
        self.alloc_type.copy_(torch.as_tensor(np.ascontiguousarray(alloc_type, np.int32)))
        self.alloc_count.copy_(torch.as_tensor(np.ascontiguousarray(alloc_count, np.int32)))
        self.load_queue(queue, priority)

    def load_queue(self, queue, priority) -> None:
        """Replace the queue, keeping the allocation on the device (synchronously)."""
        torch = self.torch
        q = np.ascontiguousarray(queue, np.int32)
        p = np.ascontiguousarray(priority, np.int32)
        if q.shape != p.shape or q.ndim != 1 or len(q) > self.n_jobs:
            raise ValueError("queue / priority must be 1-D of equal length <= n_jobs")
        self.n_queue = len(q)
        if len(q):
            self.queue[: len(q)].copy_(torch.as_tensor(q))
            self.priority[: len(q)].copy_(torch.as_tensor(p))
        torch.cuda.synchronize(self.dev)

    def step(self, depth: int, stream=None) -> None:
        """One scheduling step on the loaded state (asynchronous)."""
        s = self.torch.cuda.current_stream(self.dev) if stream is None else stream
        arena_schedule(self.ctx, self.n_jobs, self.n_types, self.n_counts, self.thr, self.counts,
                       self.capacity, self.alloc_type, self.alloc_count, self.queue, self.priority,
                       self.n_queue, depth, self.launched, self.result, s.cuda_stream,
                       self.batch, self.iters, self.deadline, self.objective)

    def results(self) -> dict:
        """Synchronise and copy the state after the last step to the host."""
        self.torch.cuda.synchronize(self.dev)
        res = self.result.cpu().numpy()
        scanned = int(np.uint32(res[5])) | (int(np.uint32(res[6])) << 32)
        return dict(status=int(res[0]), moves=[int(v) for v in res[1:4]], decisions=int(res[4]),
                    scanned=scanned,
                    alloc_type=self.alloc_type.cpu().numpy(), alloc_count=self.alloc_count.cpu().numpy(),
                    launched=self.launched[: self.n_queue].cpu().numpy())

    def close(self) -> None:
        if getattr(self, "_alive", False):
            self.torch.cuda.synchronize(self.dev)
            arena_destroy(self.ctx)
            self._alive = False

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
