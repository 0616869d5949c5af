"""Host-side checks of the C ABI (no GPU): the library loads, exports every
symbol include/arena.h declares, and rejects bad arguments before any HIP call.
Contexts are created lazily, so every call here stays on the host."""
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2403_16125_amd import arena
from paper_2403_16125_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "arena.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(arena_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    arena.load()
    out = subprocess.run(["nm", "-D", "--defined-only", arena.library_path()],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (arena_[a-z_]+)", out))
    declared = _declared()
    assert declared, "no declarations parsed"
    missing = [d for d in declared if d not in exported]
    assert not missing, missing
    assert set(arena.EXPORTED) == set(declared)


def test_status_strings():
    assert arena.arena_status_string(0) == "ARENA_OK"
    assert arena.arena_status_string(5) == "ARENA_ERR_UNSUPPORTED"
    assert "UNKNOWN" in arena.arena_status_string(99)


def test_create_destroy_null_safe():
    lib = arena.load()
    assert lib.arena_create(0, None) == arena.ARENA_ERR_INVALID_ARG
    import ctypes
    h = ctypes.c_void_p()
    assert lib.arena_create(-1, ctypes.byref(h)) == arena.ARENA_ERR_INVALID_ARG
    lib.arena_destroy(None)            # must not crash
    assert lib.arena_last_error(None) == b"no context"
    ctx = arena.arena_create(0)
    arena.arena_destroy(ctx)


@pytest.fixture
def ctx():
    c = arena.arena_create(0)
    yield c
    arena.arena_destroy(c)


def _expect(status, fn, *args, match=None, **kw):
    with pytest.raises(arena.ArenaError) as ei:
        fn(*args, **kw)
    assert ei.value.status == status, str(ei.value)
    if match:
        assert match in ei.value.message, ei.value.message


FAKE = 0x1000   # never dereferenced: validation rejects first or only host data is read


def test_bind_jobs_validation(ctx):
    off = np.array([0, 3, 5], np.int32)
    bat = np.array([8, 8], np.int32)
    args = (off, bat, FAKE, FAKE, FAKE, FAKE, FAKE)
    arena.arena_bind_jobs(ctx, *args)   # host-only: succeeds
    _expect(1, arena.arena_bind_jobs, ctx, off, bat, FAKE, 0, FAKE, FAKE, FAKE, match="per-layer")
    _expect(1, arena.arena_bind_jobs, ctx, np.array([1, 3], np.int32), bat[:1], *args[2:],
            match="layer_offset[0]")
    _expect(1, arena.arena_bind_jobs, ctx, np.array([0, 3, 3], np.int32), bat, *args[2:],
            match="0 layers")
    _expect(1, arena.arena_bind_jobs, ctx, off, np.array([8, 0], np.int32), *args[2:], match="batch")
    _expect(5, arena.arena_bind_jobs, ctx, np.array([0, 129], np.int32), bat[:1], *args[2:],
            match="129 layers")
    _expect(1, arena.arena_bind_jobs, ctx, off, bat, *args[2:], 7, match="n_layers_total")
    lib = arena.load()
    assert lib.arena_bind_jobs(ctx, None) == arena.ARENA_ERR_INVALID_ARG


def _grids(**over):
    g = dict(speed=[1.0, 0.5], mem_bytes=[4e10, 8e10], bw_intra=[3e11, 3e11], bw_inter=[2.5e10, 2.5e10],
             gpus_per_node=[4, 4], counts=[1, 2, 4, 8])
    g.update(over)
    return g


def test_bind_grids_validation(ctx):
    arena.arena_bind_grids(ctx, **_grids())
    arena.arena_bind_grids(ctx, **_grids(bw_inter=[np.inf, 1.0]))      # infinite links allowed
    _expect(1, arena.arena_bind_grids, ctx, **_grids(speed=[1.0, 0.0]), match="speed")
    _expect(1, arena.arena_bind_grids, ctx, **_grids(speed=[1.0, np.nan]), match="speed")
    _expect(1, arena.arena_bind_grids, ctx, **_grids(mem_bytes=[-1.0, 1.0]), match="mem")
    _expect(1, arena.arena_bind_grids, ctx, **_grids(bw_intra=[0.0, 1.0]), match="bandwidth")
    _expect(1, arena.arena_bind_grids, ctx, **_grids(gpus_per_node=[0, 4]), match="gpus_per_node")
    _expect(5, arena.arena_bind_grids, ctx, **_grids(gpus_per_node=[32, 4]), match="gpus_per_node")
    _expect(1, arena.arena_bind_grids, ctx, **_grids(counts=[1, 2, 2]), match="twice")
    _expect(1, arena.arena_bind_grids, ctx, **_grids(counts=[0]), match="counts")
    _expect(5, arena.arena_bind_grids, ctx, **_grids(counts=[2048]), match="max 1024")


def test_kappa_and_plan_space_validation(ctx):
    _expect(4, arena.arena_set_kappa, ctx, np.ones(8, np.float32), match="bind grids")
    arena.arena_bind_grids(ctx, **_grids())
    arena.arena_set_kappa(ctx, np.full(8, 1.5, np.float32))
    _expect(1, arena.arena_set_kappa, ctx, np.ones(7, np.float32), match="expected 8")
    _expect(1, arena.arena_set_kappa, ctx, np.array([1] * 7 + [0], np.float32), match="kappa[7]")
    _expect(1, arena.arena_set_kappa, ctx, np.array([1] * 7 + [np.inf], np.float32), match="kappa[7]")
    arena.arena_set_plan_space(ctx, [1, 2, 4], 1e-6)
    _expect(1, arena.arena_set_plan_space, ctx, [1, 2, 2], 1e-6, match="twice")
    _expect(1, arena.arena_set_plan_space, ctx, [0], 1e-6)
    _expect(5, arena.arena_set_plan_space, ctx, [128], 1e-6)
    _expect(5, arena.arena_set_plan_space, ctx, list(range(1, 18)), 1e-6)
    _expect(1, arena.arena_set_plan_space, ctx, [1], -1.0, match="tie_eps")
    _expect(1, arena.arena_set_plan_space, ctx, [1], float("nan"), match="tie_eps")


def test_estimate_not_ready_and_bad_outputs(ctx):
    _expect(4, arena.arena_estimate, ctx, FAKE, FAKE, FAKE, match="bind")
    w = wl.tiny()
    arena.arena_bind_jobs(ctx, w.layer_offset, w.batch, FAKE, FAKE, FAKE, FAKE, FAKE)
    arena.arena_bind_grids(ctx, w.speed, w.mem, w.bw_intra, w.bw_inter, w.gpus_per_node, w.counts)
    _expect(4, arena.arena_estimate, ctx, FAKE, FAKE, FAKE, match="bind")
    arena.arena_set_plan_space(ctx, w.m_values, w.tie_eps)
    _expect(1, arena.arena_estimate, ctx, FAKE, 0, FAKE, match="output")
    _expect(1, arena.arena_estimate, ctx, FAKE, FAKE, FAKE, FAKE, 5, match="cuts_stride")


def _plans_of_cell(n, G, L, Bg, ms):
    cnt = 0
    for tp in range(1, n + 1):
        if n % tp or tp > G or G % tp:
            continue
        for pp in range(1, n // tp + 1):
            if (n // tp) % pp or pp > L:
                continue
            dp = n // (tp * pp)
            cnt += sum(1 for m in ms if Bg % (dp * m) == 0)
    return cnt


@pytest.mark.parametrize("name", ["tiny", "small", "trace"])
def test_space_size_matches_enumeration(ctx, name):
    w = wl.make(name)
    arena.arena_bind_jobs(ctx, w.layer_offset, w.batch, FAKE, FAKE, FAKE, FAKE, FAKE)
    arena.arena_bind_grids(ctx, w.speed, w.mem, w.bw_intra, w.bw_inter, w.gpus_per_node, w.counts)
    arena.arena_set_plan_space(ctx, w.m_values, w.tie_eps)
    s = arena.arena_space_size_get(ctx)
    ms = [int(m) for m in w.m_values]
    total, mx = 0, 0
    cache = {}
    for j in range(w.n_jobs):
        key = (w.layers(j), int(w.batch[j]))
        if key not in cache:
            cache[key] = [[_plans_of_cell(int(n), int(G), key[0], key[1], ms) for n in w.counts]
                          for G in w.gpus_per_node]
        for row in cache[key]:
            total += sum(row)
            mx = max(mx, max(row))
    assert s["cells"] == w.n_cells
    assert s["plans"] == total
    assert s["max_plans_per_cell"] == mx
    assert s["max_layers"] == int(np.diff(w.layer_offset).max())


def test_bound_pruning_switch(ctx):
    lib = arena.load()
    assert lib.arena_set_bound_pruning(None, 1) == arena.ARENA_ERR_INVALID_ARG
    arena.arena_set_bound_pruning(ctx, False)     # any state; host only
    arena.arena_set_bound_pruning(ctx, True)


def test_partition_rule_switch(ctx):
    lib = arena.load()
    assert lib.arena_set_partition_rule(None, 0) == arena.ARENA_ERR_INVALID_ARG
    for bad in (-1, 3, 7):
        _expect(arena.ARENA_ERR_INVALID_ARG, arena.arena_set_partition_rule, ctx, bad, match="partition rule")
    arena.arena_set_partition_rule(ctx, arena.PARTITION_MEMORY)
    arena.arena_set_partition_rule(ctx, arena.PARTITION_EXACT_T)
    arena.arena_set_partition_rule(ctx, arena.PARTITION_BALANCED)
    src = open(HEADER).read()
    assert re.search(r"#define ARENA_PARTITION_BALANCED 0\b", src)
    assert re.search(r"#define ARENA_PARTITION_MEMORY 1\b", src)
    assert re.search(r"#define ARENA_PARTITION_EXACT_T 2\b", src)
    assert re.search(rf"#define ARENA_EXACT_T_MAX_LAYERS {arena.EXACT_T_MAX_LAYERS}\b", src)


def test_exact_t_refuses_long_jobs_and_comm_tables(ctx):
    # host-side: both refusals come before any device call
    w = wl.tiny()
    arena.arena_bind_grids(ctx, w.speed, w.mem, w.bw_intra, w.bw_inter, w.gpus_per_node, w.counts)
    arena.arena_set_plan_space(ctx, w.m_values, 1e-6)
    arena.arena_set_partition_rule(ctx, arena.PARTITION_EXACT_T)
    L = arena.EXACT_T_MAX_LAYERS + 1
    arena.arena_bind_jobs(ctx, np.array([0, 3, 3 + L], np.int32), np.array([8, 8], np.int32),
                          FAKE, FAKE, FAKE, FAKE, FAKE)
    _expect(arena.ARENA_ERR_UNSUPPORTED, arena.arena_estimate, ctx, FAKE, FAKE, FAKE, match="exact-T")
    arena.arena_bind_jobs(ctx, w.layer_offset, w.batch, FAKE, FAKE, FAKE, FAKE, FAKE)
    arena.arena_set_comm_tables(ctx, *wl.comm_tables(w))
    _expect(arena.ARENA_ERR_UNSUPPORTED, arena.arena_estimate, ctx, FAKE, FAKE, FAKE, match="comm tables")


def test_comm_tables_validation(ctx):
    lib = arena.load()
    assert lib.arena_set_comm_tables(None, 0, None, None) == arena.ARENA_ERR_INVALID_ARG
    good_v = np.array([[[0.0, 1e6, 1e9]] * 2], np.float64)        # 1 type x 2 links x 3 points
    good_l = np.array([[[1e-5, 2e-5, 1e-2]] * 2], np.float64)
    _expect(arena.ARENA_ERR_NOT_READY, arena.arena_set_comm_tables, ctx, good_v, good_l, match="grids")
    w = wl.tiny()
    arena.arena_bind_grids(ctx, w.speed, w.mem, w.bw_intra, w.bw_inter, w.gpus_per_node, w.counts)
    T = int(w.n_types)
    v = np.broadcast_to(good_v[0], (T, 2, 3)).copy()
    lt = np.broadcast_to(good_l[0], (T, 2, 3)).copy()
    arena.arena_set_comm_tables(ctx, v, lt)
    arena.arena_set_comm_tables(ctx)                                # back to volume / bandwidth
    bad = []
    x = v.copy(); x[0, 0, 0] = 1.0; bad.append((x, lt, "volume 0"))
    x = v.copy(); x[0, 1, 2] = x[0, 1, 1]; bad.append((x, lt, "not increasing"))
    y = lt.copy(); y[0, 0, 2] = 1e-6; bad.append((v, y, "decrease"))
    y = lt.copy(); y[0, 0, 0] = -1.0; bad.append((v, y, "negative"))
    y = lt.copy(); y[0, 0, 1] = np.nan; bad.append((v, y, "not finite"))
    for vv, ll, msg in bad:
        _expect(arena.ARENA_ERR_INVALID_ARG, arena.arena_set_comm_tables, ctx, vv, ll, match=msg)
    one_v, one_l = v[:, :, :1].copy(), lt[:, :, :1].copy()
    _expect(arena.ARENA_ERR_INVALID_ARG, arena.arena_set_comm_tables, ctx, one_v, one_l, match="points")
    many_v = np.cumsum(np.ones((T, 2, 17)), axis=2) - 1.0
    _expect(arena.ARENA_ERR_INVALID_ARG, arena.arena_set_comm_tables, ctx, many_v, np.ones((T, 2, 17)),
            match="points")
    assert lib.arena_set_comm_tables(ctx, 3, None, None) == arena.ARENA_ERR_INVALID_ARG


def test_comm_tables_rejected_with_the_memory_rule(ctx):
    # host-side: the estimate refuses the combination before touching a device
    w = wl.tiny()
    arena.arena_bind_grids(ctx, w.speed, w.mem, w.bw_intra, w.bw_inter, w.gpus_per_node, w.counts)
    arena.arena_set_plan_space(ctx, w.m_values, 1e-6)
    arena.arena_bind_jobs(ctx, w.layer_offset, w.batch, FAKE, FAKE, FAKE, FAKE, FAKE)
    arena.arena_set_comm_tables(ctx, *wl.comm_tables(w))
    arena.arena_set_partition_rule(ctx, arena.PARTITION_MEMORY)
    _expect(arena.ARENA_ERR_UNSUPPORTED, arena.arena_estimate, ctx, FAKE, FAKE, FAKE, match="comm tables")


def test_unsorted_microbatch_counts_accepted(ctx):
    # the library sorts them for the kernel; the caller's order is free
    arena.arena_set_plan_space(ctx, [8, 1, 4, 2], 1e-6)


def test_counter_struct_layout():
    # the binding's view of arena_counters matches the header's field order
    src = open(HEADER).read()
    body = re.search(r"typedef struct arena_counters \{(.*?)\} arena_counters;", src, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"int64_t\s+(\w+);", body)
    assert fields == [f for f, _ in arena.Counters._fields_]


def test_sched_desc_layout(tmp_path):
    # the binding's arena_sched_desc has the C field offsets (compiled with gcc)
    import ctypes
    names = [f for f, _ in arena.SchedDesc._fields_]
    prog = tmp_path / "off.c"
    prog.write_text("#include <stdio.h>\n#include <stddef.h>\n#include \"arena.h\"\nint main(void){\n"
                    + "".join(f'printf("%zu\\n", offsetof(arena_sched_desc, {n}));\n' for n in names)
                    + 'printf("%zu\\n", sizeof(arena_sched_desc));\nreturn 0;}\n')
    exe = tmp_path / "off"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(prog)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [getattr(arena.SchedDesc, n).offset for n in names] + [ctypes.sizeof(arena.SchedDesc)]
    assert got == want


def test_schedule_validation(ctx):
    # every case is rejected on the host before any HIP call (the pointers are
    # never dereferenced)
    lib = arena.load()
    fake = 0x1000
    base = dict(n_jobs=4, n_types=2, n_counts=3, thr=fake, counts=[1, 2, 4], capacity=[4, 4],
                alloc_type=fake, alloc_count=fake, queue=fake, priority=fake, n_queue=2, depth=4,
                launched=fake, result=fake)

    def call(**kw):
        a = dict(base, **kw)
        with pytest.raises(arena.ArenaError) as e:
            arena.arena_schedule(ctx, **a)
        return e.value.status

    assert lib.arena_schedule(None, None, None) == arena.ARENA_ERR_INVALID_ARG
    assert lib.arena_schedule(ctx, None, None) == arena.ARENA_ERR_INVALID_ARG
    assert call(n_jobs=-1) == arena.ARENA_ERR_INVALID_ARG
    assert call(n_jobs=arena.MAX_SCHED_JOBS + 1) == arena.ARENA_ERR_UNSUPPORTED
    assert call(n_types=0, capacity=[]) == arena.ARENA_ERR_INVALID_ARG
    assert call(n_types=65, capacity=[1] * 65) == arena.ARENA_ERR_UNSUPPORTED
    assert call(n_counts=0, counts=[]) == arena.ARENA_ERR_INVALID_ARG
    assert call(n_counts=513, counts=list(range(1, 514))) == arena.ARENA_ERR_UNSUPPORTED
    assert call(n_queue=5) == arena.ARENA_ERR_INVALID_ARG
    assert call(n_queue=-1) == arena.ARENA_ERR_INVALID_ARG
    assert call(depth=0) == arena.ARENA_ERR_INVALID_ARG
    assert call(depth=arena.MAX_SCHED_DEPTH + 1) == arena.ARENA_ERR_INVALID_ARG
    assert call(counts=[1, 4, 2]) == arena.ARENA_ERR_INVALID_ARG
    assert "ascending" in arena.arena_last_error(ctx)
    assert call(counts=[1, 2, 2]) == arena.ARENA_ERR_INVALID_ARG
    assert call(counts=[0, 2, 4]) == arena.ARENA_ERR_INVALID_ARG
    assert call(counts=[1, 2, 2048]) == arena.ARENA_ERR_INVALID_ARG
    assert call(capacity=[4, -1]) == arena.ARENA_ERR_INVALID_ARG
    assert call(capacity=[4, (1 << 24) + 1]) == arena.ARENA_ERR_INVALID_ARG
    assert call(thr=None) == arena.ARENA_ERR_INVALID_ARG
    assert call(result=None) == arena.ARENA_ERR_INVALID_ARG
    assert call(queue=None) == arena.ARENA_ERR_INVALID_ARG
    assert call(launched=None) == arena.ARENA_ERR_INVALID_ARG
    assert call(batch=fake) == arena.ARENA_ERR_INVALID_ARG           # deadline arrays: all or none
    assert call(batch=fake, iters=fake) == arena.ARENA_ERR_INVALID_ARG
    assert call(objective=2) == arena.ARENA_ERR_INVALID_ARG            # neither objective
    assert "objective" in arena.arena_last_error(ctx)
    assert call(objective=-1) == arena.ARENA_ERR_INVALID_ARG
    # the fairness objective needs batch and iters (a deadline is optional)
    assert call(objective=arena.SCHED_FAIRNESS) == arena.ARENA_ERR_INVALID_ARG
    assert call(objective=arena.SCHED_FAIRNESS, batch=fake) == arena.ARENA_ERR_INVALID_ARG
    assert call(objective=arena.SCHED_FAIRNESS, iters=fake, deadline=fake) == arena.ARENA_ERR_INVALID_ARG
    assert "batch and iters" in arena.arena_last_error(ctx)


def test_proxy_desc_layout(tmp_path):
    import ctypes
    names = [f for f, _ in arena.ProxyDesc._fields_]
    prog = tmp_path / "off.c"
    prog.write_text("#include <stdio.h>\n#include <stddef.h>\n#include \"arena.h\"\nint main(void){\n"
                    + "".join(f'printf("%zu\\n", offsetof(arena_proxy_desc, {n}));\n' for n in names)
                    + 'printf("%zu\\n", sizeof(arena_proxy_desc));\nreturn 0;}\n')
    exe = tmp_path / "off"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(prog)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [getattr(arena.ProxyDesc, n).offset for n in names] + [ctypes.sizeof(arena.ProxyDesc)]
    assert got == want


def test_proxy_validation(ctx):
    # rejected on the host before any HIP call (output pointers never touched)
    lib = arena.load()
    fake = 0x1000
    assert lib.arena_proxy_estimate(None, None, None, None, None, None) == arena.ARENA_ERR_INVALID_ARG
    with pytest.raises(arena.ArenaError) as e:
        arena.arena_proxy_estimate(ctx, [2e12], 1e14, 16, fake, fake, fake)
    assert e.value.status == arena.ARENA_ERR_NOT_READY
    w = wl.make("tiny")
    arena.arena_bind_jobs(ctx, w.layer_offset, w.batch, fake, fake, fake, fake, fake,
                          n_layers_total=int(w.layer_offset[-1]))
    arena.arena_bind_grids(ctx, w.speed, w.mem, w.bw_intra, w.bw_inter, w.gpus_per_node, w.counts)
    arena.arena_set_plan_space(ctx, w.m_values, 1e-6)
    hbm = w.hbm_bw()

    def status(**kw):
        a = dict(hbm_bw=hbm, f_ref=1e14, n_ops=16, t_iter=fake, thr=fake, plan=fake)
        a.update(kw)
        with pytest.raises(arena.ArenaError) as ex:
            arena.arena_proxy_estimate(ctx, a["hbm_bw"], a["f_ref"], a["n_ops"], a["t_iter"], a["thr"],
                                       a["plan"])
        return ex.value.status

    assert status(n_ops=0) == arena.ARENA_ERR_INVALID_ARG
    assert status(n_ops=17) == arena.ARENA_ERR_INVALID_ARG
    assert status(f_ref=0.0) == arena.ARENA_ERR_INVALID_ARG
    assert status(f_ref=float("inf")) == arena.ARENA_ERR_INVALID_ARG
    assert status(hbm_bw=[2e12, 0.0]) == arena.ARENA_ERR_INVALID_ARG
    assert status(hbm_bw=[2e12, float("nan")]) == arena.ARENA_ERR_INVALID_ARG
    assert status(t_iter=None) == arena.ARENA_ERR_INVALID_ARG
    assert status(plan=None) == arena.ARENA_ERR_INVALID_ARG
    assert lib.arena_proxy_estimate(ctx, None, fake, fake, fake, None) == arena.ARENA_ERR_INVALID_ARG


def _bind_host_only(ctx, n_jobs, L=4, n_types=8, n_counts=16):
    """Jobs, grids and plan space bound with fake device pointers (never read:
    every check below fails on the host first)."""
    off = (np.arange(n_jobs + 1, dtype=np.int64) * L).astype(np.int32)
    arena.arena_bind_jobs(ctx, off, np.full(n_jobs, 8, np.int32), FAKE, FAKE, FAKE, FAKE, FAKE)
    arena.arena_bind_grids(ctx, speed=[1.0] * n_types, mem_bytes=[8e10] * n_types, bw_intra=[3e11] * n_types,
                           bw_inter=[2.5e10] * n_types, gpus_per_node=[8] * n_types,
                           counts=[8 * (i + 1) for i in range(n_counts)])
    arena.arena_set_plan_space(ctx, [1, 2, 4, 8], 1e-6)


def test_workspace_limit_out_of_memory(ctx):
    """A workload whose library-owned tables exceed the context's workspace cap
    fails with OUT_OF_MEMORY before any device call (this runs without a GPU);
    a negative cap is rejected."""
    _expect(1, arena.arena_set_workspace_limit, ctx, -1, match="workspace")
    _bind_host_only(ctx, 5000)
    arena.arena_set_workspace_limit(ctx, 64 << 10)
    _expect(2, arena.arena_estimate, ctx, FAKE, FAKE, FAKE, match="limit 65536")
    # J = 5000, T = 8, NC = 16: 4 J T + 8 J + ... bytes of tables, the header's
    # formula (checked before the device is asked for its CU count, which sets
    # the size of the split caches)
    msg = None
    try:
        arena.arena_estimate(ctx, FAKE, FAKE, FAKE)
    except arena.ArenaError as e:
        msg = e.message
    need = int(re.search(r"need (\d+) bytes", msg).group(1))
    J, T, NC = 5000, 8, 16
    approx = 4 * (J + 1) + 4 * J + 40 * T + 8 * NC + 4 * T * NC + 4 * J * T
    assert approx <= need <= approx + 2560


def test_noalloc_rejects_a_workload_beyond_its_scratch(ctx):
    """The no-allocation entry point takes the same host checks as
    arena_estimate and rejects a workload whose tables exceed its static
    scratch with OUT_OF_MEMORY (here 600,000 jobs x 8 types: 24 MB of tables),
    before any device call."""
    _expect(4, arena.arena_estimate_noalloc, ctx, FAKE, FAKE, FAKE, match="bind")
    _bind_host_only(ctx, 600_000)
    _expect(1, arena.arena_estimate_noalloc, ctx, FAKE, 0, FAKE, match="output")
    _expect(2, arena.arena_estimate_noalloc, ctx, FAKE, FAKE, FAKE, match="scratch")
    assert arena.NOALLOC_SCRATCH_BYTES == 16 << 20
