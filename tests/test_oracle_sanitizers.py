"""The C oracles and the host side of the C ABI under the sanitizers (CPU only).

* UndefinedBehaviorSanitizer: both oracles are rebuilt with
  -fsanitize=undefined (every report fatal) and the oracle pin suites run
  against those copies in a child process.
* AddressSanitizer + UBSan: a driver executable links the oracle sources and
  evaluates whole workloads (tiny, small, the edge shapes, sampled trace-like
  and MoE cells; balanced, memory and exact-T rules, communication tables,
  the proxy planner) from input arrays allocated to their exact sizes; its outputs must
  equal, bit for bit, those of the regular build loaded in this process.
* AddressSanitizer + UBSan on the host side of the library: arena_host.cpp
  built with g++ (no device code: the kernel launchers are stubs that report
  no device) and driven through every validation path of the ABI.
"""
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

from paper_2403_16125_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fno-sanitize-recover=all"]
SAN_ENV = dict(os.environ, UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1")

needs_gcc = pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None,
                               reason="gcc/g++ not available")


@needs_gcc
def test_oracle_pins_under_ubsan(tmp_path):
    from oracle import oracle as oracle_c
    from oracle import proxy as proxy_c
    lib = oracle_c.build(out=str(tmp_path / "liboracle_ubsan.so"), extra_flags=SAN + ["-fsanitize=undefined"])
    plib = proxy_c.build(out=str(tmp_path / "libproxy_ubsan.so"), extra_flags=SAN + ["-fsanitize=undefined"])
    pins = ["test_oracle_partition.py", "test_oracle_pricing.py", "test_oracle_memory_partition.py",
            "test_oracle_comm_tables.py", "test_oracle_proxy.py", "test_oracle_exact_t.py"]
    pins = [os.path.join(HERE, f) for f in pins if os.path.exists(os.path.join(HERE, f))]
    env = dict(SAN_ENV, ARENA_ORACLE_LIB=lib, ARENA_PROXY_ORACLE_LIB=plib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"]
                       + pins, cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    out = r.stdout + r.stderr
    assert "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]


def _edge():
    rng = np.random.default_rng(5)
    jobs = [dict(t=[2e-3], p=[1e8], a=[1e6], x=[1e5], a2a=[0.0], batch=8),
            dict(t=[0.0, 1e-3, 0.0, 0.0, 2e-3], p=[1e8] * 5, a=[1e6] * 5, x=[1e5] * 5, a2a=[0.0] * 5,
                 batch=16),
            dict(t=list(rng.lognormal(-6, 0.8, 128)), p=list(rng.uniform(1e8, 3e8, 128)), a=[4e6] * 128,
                 x=[2.5e5] * 128, a2a=[0.0 if i % 2 == 0 else 4e5 for i in range(128)], batch=128),
            dict(t=[1e-3] * 24, p=[1e10] * 24, a=[1e9] * 24, x=[1e7] * 24, a2a=[0.0] * 24, batch=4)]
    types = [dict(speed=1.0, mem=80e9, bw_intra=300e9, bw_inter=25e9, gpus_per_node=8),
             dict(speed=0.5, mem=16e9, bw_intra=np.inf, bw_inter=np.inf, gpus_per_node=1),
             dict(speed=0.7, mem=40e9, bw_intra=64e9, bw_inter=12.5e9, gpus_per_node=16)]
    counts = [1, 2, 3, 8, 24, 128]
    return wl.from_lists(jobs, types, counts, [1, 2, 4, 8, 16, 32, 64],
                         kappa=rng.uniform(1.0, 2.0, len(types) * len(counts)))


def _request(path, kind, rule, w, ids, tables=None, stride=128, n_ops=16, f_ref=1e14):
    K = 0 if tables is None else int(np.asarray(tables[0]).shape[2])
    with open(path, "wb") as fh:
        np.asarray([kind, rule if kind != 2 else n_ops, w.n_jobs, len(w.t), w.n_types, w.n_counts,
                    len(w.m_values), len(ids), K, stride], np.int32).tofile(fh)
        np.asarray([w.tie_eps, f_ref], np.float64).tofile(fh)
        for v, dt in ((w.layer_offset, np.int32), (w.t, np.float32), (w.p, np.float32), (w.a, np.float32),
                      (w.x, np.float32), (w.a2a, np.float32), (w.batch, np.int32), (w.speed, np.float32),
                      (w.mem, np.float32), (w.bw_intra, np.float32), (w.bw_inter, np.float32),
                      (w.gpus_per_node, np.int32), (w.hbm_bw(), np.float32), (w.counts, np.int32),
                      (np.asarray(w.kappa)[0], np.float32), (w.m_values, np.int32), (ids, np.int64)):
            np.ascontiguousarray(v, dt).tofile(fh)
        if tables is not None:
            np.ascontiguousarray(tables[0], np.float64).tofile(fh)
            np.ascontiguousarray(tables[1], np.float64).tofile(fh)


@needs_gcc
def test_oracles_under_asan_match_the_regular_build(tmp_path):
    from oracle import oracle as oracle_c
    from oracle import proxy as proxy_c
    exe = str(tmp_path / "oracle_asan")
    subprocess.run(["gcc", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-Wall"] + SAN +
                   ["-fsanitize=address,undefined", "-o", exe, os.path.join(HERE, "oracle_asan_driver.c"),
                    os.path.join(ROOT, "oracle", "arena_oracle.c"), os.path.join(ROOT, "oracle", "proxy_oracle.c"),
                    "-lm"], check=True)
    rng = np.random.default_rng(17)
    cases = []
    for name in ("tiny", "small"):
        w = wl.make(name)
        cases.append((name, w, np.arange(w.n_cells, dtype=np.int64)))
    e = _edge()
    cases.append(("edge", e, np.arange(e.n_cells, dtype=np.int64)))
    for name, k in (("trace", 60), ("moe", 12)):
        w = wl.make(name)
        cases.append((name, w, np.sort(rng.choice(w.n_cells, k, replace=False)).astype(np.int64)))
    runs = []
    for name, w, ids in cases:
        runs.append((f"{name} balanced", 0, 0, w, ids, None))
    runs.append(("small memory rule", 0, 1, cases[1][1], cases[1][2][::3], None))
    runs.append(("edge memory rule", 0, 1, e, cases[2][2], None))
    runs.append(("small exact-T", 0, 2, cases[1][1], cases[1][2][::97], None))
    runs.append(("trace exact-T", 0, 2, cases[3][1], cases[3][2][:6], None))
    runs.append(("small tables", 1, 0, cases[1][1], cases[1][2][::5], wl.comm_tables(cases[1][1])))
    runs.append(("edge tables", 1, 0, e, cases[2][2], wl.comm_tables(e)))
    runs.append(("small proxy", 2, 0, cases[1][1], cases[1][2][::4], None))
    runs.append(("edge proxy", 2, 0, e, cases[2][2], None))
    for label, kind, rule, w, ids, tables in runs:
        req, out = str(tmp_path / "req.bin"), str(tmp_path / "out.bin")
        _request(req, kind, rule, w, ids, tables)
        r = subprocess.run([exe, req, out], env=SAN_ENV, capture_output=True, text=True, timeout=900)
        assert r.returncode == 0, f"{label}: rc {r.returncode}\n{r.stderr[-4000:]}"
        assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
        raw = np.fromfile(out, np.uint8)
        n = len(ids)
        if kind in (0, 1):
            ref = (oracle_c.cells(w, ids, rule=rule) if kind == 0 else oracle_c.cells_tab(w, ids, tables))
            res = raw[:16 * n].view(np.float64).reshape(n, 2)
            o = 16 * n
            plan = raw[o:o + 16 * n].view(np.int32).reshape(n, 4)
            o += 16 * n
            cuts = raw[o:o + 4 * n * 128].view(np.int32).reshape(n, 128)
            o += 4 * n * 128
            nplans = raw[o:o + 4 * n].view(np.int32)
            assert np.array_equal(res[:, 0].view(np.int64), ref["T"].view(np.int64)), label
            assert np.array_equal(res[:, 1].view(np.int64), ref["thr"].view(np.int64)), label
            assert np.array_equal(plan, np.stack([ref["dp"], ref["tp"], ref["pp"], ref["m"]], 1)), label
            assert np.array_equal(cuts, ref["cuts"]), label
            assert np.array_equal(nplans, ref["nplans"]), label
        else:
            ref = proxy_c.cells(w, ids)
            o4 = raw[:32 * n].view(np.float64).reshape(n, 4)
            assert np.array_equal(o4[:, 0].view(np.int64), ref["T"].view(np.int64)), label
            assert np.array_equal(o4[:, 3].view(np.int64), ref["thr"].view(np.int64)), label
            plan = raw[32 * n:].view(np.int32).reshape(n, 52)
            assert np.array_equal(plan[:, 0], ref["s"]) and np.array_equal(plan[:, 2:19], ref["bounds"]), label


HOST_DRIVER = r"""
#include <cmath>
#include <cstdio>
#include <cstring>
#include <vector>
#include "arena.h"

static int failures = 0;
#define EXPECT(call, want)                                                                  \
    do {                                                                                    \
        arena_status got_ = (call);                                                         \
        if (got_ != (want)) {                                                               \
            std::fprintf(stderr, "line %d: %s -> %d, want %d (%s)\n", __LINE__, #call, (int)got_, \
                         (int)(want), ctx ? arena_last_error(ctx) : "");                    \
            ++failures;                                                                     \
        }                                                                                   \
    } while (0)

int main()
{
    arena_ctx* ctx = nullptr;
    EXPECT(arena_create(-1, &ctx), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_create(0, nullptr), ARENA_ERR_INVALID_ARG);
    arena_destroy(nullptr);
    EXPECT(arena_create(0, &ctx), ARENA_OK);
    float* F = (float*)0x1000;        // never dereferenced on the host
    uint32_t* P = (uint32_t*)0x1000;
    EXPECT(arena_estimate(ctx, F, F, P, nullptr, 0, nullptr), ARENA_ERR_NOT_READY);
    EXPECT(arena_estimate_noalloc(ctx, F, F, P, nullptr, 0, nullptr), ARENA_ERR_NOT_READY);
    EXPECT(arena_bind_jobs(ctx, nullptr), ARENA_ERR_INVALID_ARG);
    const int J = 50000;
    std::vector<int32_t> off(J + 1), bat(J, 64);
    for (int j = 0; j <= J; ++j) off[j] = 12 * j;
    arena_jobs_desc jd{J, 12 * J, off.data(), bat.data(), F, F, F, F, F};
    EXPECT(arena_bind_jobs(ctx, &jd), ARENA_OK);
    off[J] = 12 * J + 1;
    EXPECT(arena_bind_jobs(ctx, &jd), ARENA_ERR_INVALID_ARG);
    off[J] = 12 * J;
    off[1] = 0;
    EXPECT(arena_bind_jobs(ctx, &jd), ARENA_ERR_INVALID_ARG);
    off[1] = 200;
    EXPECT(arena_bind_jobs(ctx, &jd), ARENA_ERR_UNSUPPORTED);
    off[1] = 12;
    bat[7] = 0;
    EXPECT(arena_bind_jobs(ctx, &jd), ARENA_ERR_INVALID_ARG);
    bat[7] = 64;
    EXPECT(arena_bind_jobs(ctx, &jd), ARENA_OK);
    const int T = 8, NC = 131;
    std::vector<float> speed(T, 1.0f), mem(T, 8e10f), bwi(T, 3e11f), bwe(T, 2.5e10f);
    std::vector<int32_t> gpn(T, 8), counts(NC);
    for (int i = 0; i < NC; ++i) counts[i] = i < 3 ? (1 << i) : 8 * (i - 2);
    arena_grids_desc gd{T, speed.data(), mem.data(), bwi.data(), bwe.data(), gpn.data(), NC, counts.data()};
    EXPECT(arena_set_kappa(ctx, speed.data(), T), ARENA_ERR_NOT_READY);
    speed[3] = NAN;
    EXPECT(arena_bind_grids(ctx, &gd), ARENA_ERR_INVALID_ARG);
    speed[3] = 1.0f;
    gpn[2] = 40;
    EXPECT(arena_bind_grids(ctx, &gd), ARENA_ERR_UNSUPPORTED);
    gpn[2] = 8;
    counts[5] = counts[6];
    EXPECT(arena_bind_grids(ctx, &gd), ARENA_ERR_INVALID_ARG);
    counts[5] = 24;
    EXPECT(arena_bind_grids(ctx, &gd), ARENA_OK);
    std::vector<float> kap((size_t)T * NC, 1.25f);
    EXPECT(arena_set_kappa(ctx, kap.data(), T * NC - 1), ARENA_ERR_INVALID_ARG);
    kap[17] = -1.0f;
    EXPECT(arena_set_kappa(ctx, kap.data(), T * NC), ARENA_ERR_INVALID_ARG);
    kap[17] = 1.5f;
    EXPECT(arena_set_kappa(ctx, kap.data(), T * NC), ARENA_OK);
    int32_t ms[7] = {1, 2, 4, 8, 16, 32, 64};
    EXPECT(arena_set_plan_space(ctx, ms, 0, 1e-6), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_set_plan_space(ctx, ms, 7, -1.0), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_set_plan_space(ctx, ms, 7, 1e-6), ARENA_OK);
    arena_space_size sz;
    EXPECT(arena_space_size_get(ctx, &sz), ARENA_OK);
    if (sz.cells != (int64_t)J * T * NC) { std::fprintf(stderr, "cells %lld\n", (long long)sz.cells); ++failures; }
    EXPECT(arena_set_partition_rule(ctx, 7), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_set_partition_rule(ctx, ARENA_PARTITION_MEMORY), ARENA_OK);
    std::vector<double> vol((size_t)T * 2 * 3), lat((size_t)T * 2 * 3);
    for (int q = 0; q < T * 2; ++q)
        for (int k = 0; k < 3; ++k) { vol[q * 3 + k] = k * 1e6; lat[q * 3 + k] = k * 1e-3; }
    EXPECT(arena_set_comm_tables(ctx, 1, vol.data(), lat.data()), ARENA_ERR_INVALID_ARG);
    lat[4] = -1.0;
    EXPECT(arena_set_comm_tables(ctx, 3, vol.data(), lat.data()), ARENA_ERR_INVALID_ARG);
    lat[4] = 1e-3;
    EXPECT(arena_set_comm_tables(ctx, 3, vol.data(), lat.data()), ARENA_OK);
    EXPECT(arena_estimate(ctx, F, F, P, nullptr, 0, nullptr), ARENA_ERR_UNSUPPORTED);
    EXPECT(arena_set_comm_tables(ctx, 0, nullptr, nullptr), ARENA_OK);
    EXPECT(arena_estimate(ctx, F, nullptr, P, nullptr, 0, nullptr), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_estimate(ctx, F, F, P, (uint8_t*)F, 3, nullptr), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_set_workspace_limit(ctx, -5), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_set_workspace_limit(ctx, 1 << 20), ARENA_OK);
    EXPECT(arena_estimate(ctx, F, F, P, nullptr, 0, nullptr), ARENA_ERR_OUT_OF_MEMORY);
    // 50,000 jobs x 8 types: 1.6 MB of work order fit the scratch; the 24 MB
    // of tables of 600,000 do not (refused before the device is asked anything)
    const int J2 = 600000;
    std::vector<int32_t> off2(J2 + 1), bat2(J2, 64);
    for (int j = 0; j <= J2; ++j) off2[j] = 4 * j;
    arena_jobs_desc jd2{J2, 4 * J2, off2.data(), bat2.data(), F, F, F, F, F};
    EXPECT(arena_bind_jobs(ctx, &jd2), ARENA_OK);
    EXPECT(arena_estimate_noalloc(ctx, F, F, P, nullptr, 0, nullptr), ARENA_ERR_OUT_OF_MEMORY);
    EXPECT(arena_estimate(ctx, F, F, P, nullptr, 0, nullptr), ARENA_ERR_OUT_OF_MEMORY);
    arena_counters cn;
    EXPECT(arena_get_counters(ctx, &cn), ARENA_ERR_NOT_READY);
    EXPECT(arena_get_counters(ctx, nullptr), ARENA_ERR_INVALID_ARG);
    arena_sched_desc sd;
    std::memset(&sd, 0, sizeof(sd));
    EXPECT(arena_schedule(ctx, &sd, nullptr), ARENA_ERR_INVALID_ARG);
    EXPECT(arena_schedule(ctx, nullptr, nullptr), ARENA_ERR_INVALID_ARG);
    arena_proxy_desc pd{nullptr, 1e14, 16};
    EXPECT(arena_proxy_estimate(ctx, &pd, F, F, (uint64_t*)F, nullptr), ARENA_ERR_INVALID_ARG);
    std::printf("arena_status_string(5) = %s\n", arena_status_string(ARENA_ERR_UNSUPPORTED));
    arena_destroy(ctx);
    std::printf("%d failures\n", failures);
    return failures ? 1 : 0;
}
"""

HOST_STUBS = r"""
#include "arena_internal.h"
// Launchers of the host-only build: no device code is linked, every launch
// reports that there is no device (the validation paths return earlier).
namespace arena {
hipError_t launch_estimate(const EstimateArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_schedule(const SchedArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_proxy(const ProxyArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_zero_counters(unsigned long long*, int, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_validate(const ValidateArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t scratch_address(int, void**) { return hipErrorNoDevice; }
}
"""


@needs_gcc
def test_host_validation_under_asan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2403_16125_amd", "csrc")
    (tmp_path / "driver.cpp").write_text(HOST_DRIVER)
    (tmp_path / "stubs.cpp").write_text(HOST_STUBS)
    exe = str(tmp_path / "host_asan")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(rocm, "include"),
           "-I", os.path.join(ROOT, "include"), "-I", csrc] + SAN + ["-fsanitize=address,undefined",
           "-o", exe, str(tmp_path / "driver.cpp"), str(tmp_path / "stubs.cpp"),
           os.path.join(csrc, "arena_host.cpp"), "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath," + os.path.join(rocm, "lib")]
    b = subprocess.run(cmd, capture_output=True, text=True)
    if b.returncode != 0 and "amdhip64" in b.stderr:
        pytest.skip("HIP runtime library not linkable here")
    assert b.returncode == 0, b.stderr[-4000:]
    # the HIP runtime is not instrumented: leaks it keeps for the process's life are not ours
    supp = tmp_path / "lsan.supp"
    supp.write_text("leak:libamdhip64\nleak:libhsa-runtime64\nleak:libdrm\n")
    env = dict(SAN_ENV, LSAN_OPTIONS=f"suppressions={supp}")
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=300)
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "0 failures" in r.stdout
