"""Seeded synthetic workloads for the plan-space estimator.

This module only draws inputs: profiled jobs (per-layer costs and sizes),
GPU types, GPU counts, microbatch choices and per-grid contention factors.
It contains none of the estimator's arithmetic, and it is the only code that
the HIP path and the CPU oracle share.

The shapes follow the paper's workloads: transformer-like stacks of clustered
operators (Sec. 3.3 footnote on clustering), per-operator profiled latencies
and sizes (Sec. 3.4), GPU types with different speed, memory, node size and
links (Table 1), global batch sizes and model sizes of Table 2, and sequence
length 1024 (Sec. 5.1).  The production traces the paper schedules (Philly,
Helios, PAI) are not available; the "trace" and "full" workloads stand in for
them with the stated size ranges only.

Random numbers: SplitMix64 (Steele, Lea, Flood 2014) as a counter-based
stream, uniforms from the top 53 bits, normals by Box-Muller.  Every job owns
its own stream, seeded from the workload seed, so the draw of a job does not
depend on how many numbers the other jobs drew.

Units: seconds, bytes, bytes/second.  1 GB = 1e9 B.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

_MASK64 = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15

SEQ_LEN = 1024          # tokens per sample (Sec. 5.1)
F_REF = 1.0e14          # FLOP/s of a speed-1.0 GPU, converts FLOPs to seconds
HBM_REF = 2.0e12        # memory bandwidth of a speed-1.0 GPU, bytes/s (scaled by speed per type)
BASE_SEED = 240316125   # workloads use BASE_SEED + index


def _mix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


class SplitMix64:
    """Counter-based SplitMix64: draw k is mix(seed + (k+1)*gamma) mod 2^64."""

    def __init__(self, seed: int):
        self.state = int(seed) & _MASK64

    def u64(self, k: int) -> np.ndarray:
        ks = np.arange(1, k + 1, dtype=np.uint64)
        with np.errstate(over="ignore"):
            z = np.uint64(self.state) + ks * np.uint64(_GAMMA)
            out = _mix64(z)
        self.state = (self.state + k * _GAMMA) & _MASK64
        return out

    def uniform(self, k: int) -> np.ndarray:
        """k doubles in [0, 1)."""
        return (self.u64(k) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)

    def uniform_range(self, lo: float, hi: float, k: int) -> np.ndarray:
        return lo + (hi - lo) * self.uniform(k)

    def integers(self, lo: int, hi: int, k: int) -> np.ndarray:
        """k integers uniform on {lo, ..., hi}."""
        return lo + np.floor(self.uniform(k) * (hi - lo + 1)).astype(np.int64)

    def choice(self, values, k: int) -> np.ndarray:
        vals = np.asarray(values)
        return vals[np.floor(self.uniform(k) * len(vals)).astype(np.int64)]

    def normal(self, k: int) -> np.ndarray:
        """Box-Muller: one normal per pair of uniforms (cosine branch)."""
        u = self.uniform(2 * k)
        u1 = 1.0 - u[0::2]          # (0, 1]
        u2 = u[1::2]
        return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2)


def _stream(seed: int, index: int) -> SplitMix64:
    """An independent stream for item `index` of a workload with `seed`."""
    base = SplitMix64(seed)
    base.state = (base.state + index * 0xD1B54A32D192ED03) & _MASK64
    key = int(base.u64(1)[0])
    return SplitMix64(key)


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    # jobs: CSR over layers
    layer_offset: np.ndarray   # int32 [J+1]
    t: np.ndarray              # f32 [sum L] fwd+bwd seconds, whole global batch, speed-1.0 GPU
    p: np.ndarray              # f32 [sum L] parameter bytes
    a: np.ndarray              # f32 [sum L] stored activation bytes per sample
    x: np.ndarray              # f32 [sum L] boundary (output) activation bytes per sample
    a2a: np.ndarray            # f32 [sum L] all-to-all bytes per sample (0 on dense layers)
    batch: np.ndarray          # int32 [J] global batch size
    # GPU types
    speed: np.ndarray          # f32 [T] relative speed (1.0 = reference)
    mem: np.ndarray            # f32 [T] bytes per GPU
    bw_intra: np.ndarray       # f32 [T] bytes/s inside a node
    bw_inter: np.ndarray       # f32 [T] bytes/s across nodes
    gpus_per_node: np.ndarray  # int32 [T]
    # grid counts and plan space
    counts: np.ndarray         # int32 [NC]
    m_values: np.ndarray       # int32 [NM]
    kappa: np.ndarray          # f32 [R, T*NC] per-grid contention factor per round
    tie_eps: float = 1e-6
    hbm: np.ndarray | None = None   # f32 [T] memory bandwidth bytes/s (roofline loads); None: HBM_REF * speed

    def hbm_bw(self) -> np.ndarray:
        if self.hbm is not None:
            return np.asarray(self.hbm, np.float32)
        return (HBM_REF * self.speed.astype(np.float64)).astype(np.float32)

    @property
    def n_jobs(self) -> int:
        return int(self.batch.shape[0])

    @property
    def n_types(self) -> int:
        return int(self.speed.shape[0])

    @property
    def n_counts(self) -> int:
        return int(self.counts.shape[0])

    @property
    def n_cells(self) -> int:
        return self.n_jobs * self.n_types * self.n_counts

    @property
    def n_rounds(self) -> int:
        return int(self.kappa.shape[0])

    def layers(self, j: int) -> int:
        return int(self.layer_offset[j + 1] - self.layer_offset[j])

    def job_slice(self, j: int) -> slice:
        return slice(int(self.layer_offset[j]), int(self.layer_offset[j + 1]))

    def subset_jobs(self, jobs) -> "Workload":
        """A workload holding only the listed jobs (same grids and rounds)."""
        jobs = [int(j) for j in jobs]
        off = [0]
        parts = {k: [] for k in ("t", "p", "a", "x", "a2a")}
        for j in jobs:
            s = self.job_slice(j)
            for k in parts:
                parts[k].append(getattr(self, k)[s])
            off.append(off[-1] + (s.stop - s.start))
        cat = {k: (np.concatenate(v) if v else np.zeros(0, np.float32)).astype(np.float32)
               for k, v in parts.items()}
        return dataclasses.replace(
            self, name=f"{self.name}[{len(jobs)} jobs]",
            layer_offset=np.asarray(off, np.int32), batch=self.batch[jobs].astype(np.int32),
            **cat)


# ---------------------------------------------------------------- job drawing

def _pack(jobs):
    """jobs: list of dicts with per-layer float64 arrays and 'batch'."""
    off = np.zeros(len(jobs) + 1, np.int64)
    for i, jb in enumerate(jobs):
        off[i + 1] = off[i] + len(jb["t"])
    arrs = {}
    for k in ("t", "p", "a", "a2a"):
        arrs[k] = np.concatenate([jb[k] for jb in jobs]).astype(np.float32)
    # boundary tensor is 1/16 of the stored activation (a power of two: exact in f32)
    xs = []
    for jb in jobs:
        xs.append(jb["x"] if "x" in jb else jb["a"] / 16.0)
    arrs["x"] = np.concatenate(xs).astype(np.float32)
    batch = np.asarray([jb["batch"] for jb in jobs], np.int32)
    return off.astype(np.int32), arrs, batch


def _job_uniform_sizes(rng: SplitMix64, L: int, bg: int, t_kind: str):
    if t_kind == "uniform":
        t = rng.uniform_range(1e-3, 5e-3, L)
    else:  # lognormal(ln 3 ms, 0.5)
        t = np.exp(math.log(3e-3) + 0.5 * rng.normal(L))
    p = rng.uniform_range(50e6, 150e6, L)
    a = rng.uniform_range(20e6, 60e6, L)
    return dict(t=t, p=p, a=a, a2a=np.zeros(L), batch=bg)


def _job_trace(rng: SplitMix64):
    """GPT-like job: model size lognormal over 0.3-70 B params (Table 2 span)."""
    L = int(rng.integers(24, 96, 1)[0])
    bg = int(rng.choice([128, 256, 512], 1)[0])
    lo, hi = math.log(3e8), math.log(7e10)
    lnP = (lo + hi) / 2 + (hi - lo) / 4 * rng.normal(1)[0]
    P = math.exp(min(max(lnP, lo), hi))
    pi = P / L                                        # params per layer
    h = 64 * max(1, int(round(math.sqrt(pi / 12.0) / 64.0)))
    jitter = rng.uniform_range(-0.2, 0.2, L)
    t = 6.0 * pi * bg * SEQ_LEN / F_REF * (1.0 + jitter)
    p = np.full(L, 4.0 * pi)
    a = np.full(L, 64.0 * SEQ_LEN * h)
    return dict(t=t, p=p, a=a, a2a=np.zeros(L), batch=bg)


def _job_moe(rng: SplitMix64):
    """GShard-like job: 128 layers, odd layers are MoE (3x cost) with all-to-all."""
    L = 128
    h = int(rng.choice([1024, 2048, 4096], 1)[0])
    bg = int(rng.choice([256, 512, 1024], 1)[0])
    tau = 6.0 * 12.0 * h * h * bg * SEQ_LEN / F_REF
    t = np.exp(math.log(tau) + 0.8 * rng.normal(L))
    moe = (np.arange(L) % 2) == 1
    t[moe] *= 3.0
    p_dense = 4.0 * 12.0 * h * h
    a_dense = 64.0 * SEQ_LEN * h
    p = np.where(moe, 3.0 * p_dense, p_dense)
    a = np.where(moe, 3.0 * a_dense, a_dense)
    x = np.full(L, a_dense / 16.0)
    a2a = np.where(moe, SEQ_LEN * h * 2.0, 0.0)
    return dict(t=t, p=p, a=a, x=x, a2a=a2a, batch=bg)


def _pow2_upto(n):
    out, v = [], 1
    while v <= n:
        out.append(v)
        v *= 2
    return out


def _kappa(seed: int, n_grids: int, lo: float, hi: float, rounds: int) -> np.ndarray:
    out = np.empty((rounds, n_grids), np.float32)
    for r in range(rounds):
        rng = SplitMix64(seed * 1000 + r)
        out[r] = rng.uniform_range(lo, hi, n_grids).astype(np.float32)
    return out


def _build(name, seed, jobs, speed, mem_gb, bwi_gbs, bwe_gbs, gpn, counts, m_values, kappa):
    off, arrs, batch = _pack(jobs)
    return Workload(
        name=name, seed=seed, layer_offset=off, batch=batch, **arrs,
        speed=np.asarray(speed, np.float32),
        mem=(np.asarray(mem_gb, np.float64) * 1e9).astype(np.float32),
        bw_intra=(np.asarray(bwi_gbs, np.float64) * 1e9).astype(np.float32),
        bw_inter=(np.asarray(bwe_gbs, np.float64) * 1e9).astype(np.float32),
        gpus_per_node=np.asarray(gpn, np.int32),
        counts=np.asarray(counts, np.int32), m_values=np.asarray(m_values, np.int32),
        kappa=kappa)


def tiny(seed: int = BASE_SEED + 0) -> Workload:
    """4 jobs x 2 types x counts {1,2,4,8}; L=12, Bg=32, m in {1,2,4,8}."""
    jobs = [_job_uniform_sizes(_stream(seed, j), 12, 32, "uniform") for j in range(4)]
    counts = [1, 2, 4, 8]
    return _build("tiny", seed, jobs, [1.0, 0.5], [40, 80], [300, 300], [25, 25], [4, 4],
                  counts, [1, 2, 4, 8], np.ones((1, 2 * len(counts)), np.float32))


def small(seed: int = BASE_SEED + 1) -> Workload:
    """64 jobs, L in 12..48, lognormal costs; 3 types; counts 1..64 (pow2); m 1..32."""
    jobs = []
    for j in range(64):
        rng = _stream(seed, j)
        L = int(rng.integers(12, 48, 1)[0])
        bg = int(rng.choice([64, 128, 256], 1)[0])
        jobs.append(_job_uniform_sizes(rng, L, bg, "lognormal"))
    counts = _pow2_upto(64)
    return _build("small", seed, jobs, [1.0, 0.6, 0.35], [32, 40, 80], [300] * 3, [25] * 3,
                  [8] * 3, counts, _pow2_upto(32), np.ones((1, 3 * len(counts)), np.float32))


def _trace_counts(top):
    return [1, 2, 4] + list(range(8, top + 1, 8))


def trace(seed: int = BASE_SEED + 2, n_jobs: int = 1024) -> Workload:
    """GPT-like jobs (0.3-70 B params), 4 types, counts {1,2,4} + multiples of 8 to 256."""
    jobs = [_job_trace(_stream(seed, j)) for j in range(n_jobs)]
    counts = _trace_counts(256)
    kappa = _kappa(seed, 4 * len(counts), 1.0, 1.5, 1)
    return _build("trace", seed, jobs, [1.0, 0.7, 0.45, 0.25], [24, 40, 80, 96],
                  [300, 32, 300, 32], [25, 25, 12.5, 12.5], [8] * 4,
                  counts, _pow2_upto(64), kappa)


def moe(seed: int = BASE_SEED + 3, n_jobs: int = 4096) -> Workload:
    """MoE jobs (L=128, every other layer MoE), 6 types, counts 1..512 (pow2)."""
    jobs = [_job_moe(_stream(seed, j)) for j in range(n_jobs)]
    counts = _pow2_upto(512)
    return _build("moe", seed, jobs, [1.0, 0.8, 0.6, 0.45, 0.3, 0.2], [80, 96, 48, 40, 32, 24],
                  [300, 300, 32, 300, 32, 32], [25, 25, 25, 12.5, 12.5, 12.5], [8] * 6,
                  counts, _pow2_upto(64), np.ones((1, 6 * len(counts)), np.float32))


def full(seed: int = BASE_SEED + 4, n_jobs: int = 16384, rounds: int = 10) -> Workload:
    """A full scheduling round: trace-like and MoE jobs mixed 70/30 over 8 types x 131 counts,
    per-grid contention factors redrawn every round."""
    jobs = []
    for j in range(n_jobs):
        rng = _stream(seed, j)
        kind = rng.uniform(1)[0]
        jobs.append(_job_trace(rng) if kind < 0.7 else _job_moe(rng))
    counts = _trace_counts(1024)
    kappa = _kappa(seed, 8 * len(counts), 1.0, 2.0, rounds)
    return _build("full", seed, jobs, [1.0, 0.85, 0.7, 0.55, 0.45, 0.35, 0.25, 0.15],
                  [96, 80, 80, 48, 40, 48, 24, 32], [300, 300, 300, 32, 300, 32, 32, 300],
                  [25, 25, 12.5, 25, 12.5, 25, 12.5, 12.5], [8, 16, 4, 2, 2, 16, 8, 4],
                  counts, _pow2_upto(64), kappa)


WORKLOADS = {"tiny": tiny, "small": small, "trace": trace, "moe": moe, "full": full}


def make(name: str, **kw) -> Workload:
    return WORKLOADS[name](**kw)


def from_lists(jobs, types, counts, m_values, kappa=None, tie_eps: float = 1e-6,
               name: str = "explicit") -> Workload:
    """A workload from explicit values.

    jobs: list of dicts with per-layer lists t, p, a, x, a2a and an int 'batch';
    types: list of dicts with speed, mem, bw_intra, bw_inter, gpus_per_node;
    kappa: None (all 1), a scalar, or an array of shape [T*NC] or [R, T*NC]."""
    off = [0]
    cols = {k: [] for k in ("t", "p", "a", "x", "a2a")}
    for jb in jobs:
        L = len(jb["t"])
        for k in cols:
            cols[k].extend(float(v) for v in jb[k])
            assert len(jb[k]) == L
        off.append(off[-1] + L)
    nt, nc = len(types), len(counts)
    if kappa is None:
        kap = np.ones((1, nt * nc), np.float32)
    else:
        kap = np.asarray(kappa, np.float32)
        if kap.ndim == 0:
            kap = np.full((1, nt * nc), float(kap), np.float32)
        elif kap.ndim == 1:
            kap = kap.reshape(1, -1)
    f = lambda key: np.asarray([ty[key] for ty in types], np.float32)
    return Workload(
        name=name, seed=0, layer_offset=np.asarray(off, np.int32),
        **{k: np.asarray(v, np.float32) for k, v in cols.items()},
        batch=np.asarray([jb["batch"] for jb in jobs], np.int32),
        speed=f("speed"), mem=f("mem"), bw_intra=f("bw_intra"), bw_inter=f("bw_inter"),
        gpus_per_node=np.asarray([ty["gpus_per_node"] for ty in types], np.int32),
        counts=np.asarray(counts, np.int32), m_values=np.asarray(m_values, np.int32),
        kappa=kap, tie_eps=tie_eps)


# ------------------------------------------------------------ synthetic profiled communication

COMM_VOLUMES = (0.0, 65536.0, 1048576.0, 16777216.0, 268435456.0, 4294967296.0)


def comm_tables(w, volumes=COMM_VOLUMES, alpha=(1e-5, 2.5e-5), half=(262144.0, 1048576.0)):
    """Synthetic stand-ins for profiled (volume, latency) samples of each GPU
    type's intra-node (link 0) and inter-node (link 1) links: at volume v the
    latency is alpha + v / (bw * v / (v + half)), i.e. a start-up cost plus the
    volume over a bandwidth that small messages reach only in part.  Returns
    (vol, lat), each float64 [n_types][2][K]."""
    T, K = int(w.n_types), len(volumes)
    vol = np.zeros((T, 2, K), np.float64)
    lat = np.zeros((T, 2, K), np.float64)
    for g in range(T):
        for link, bw in enumerate((float(w.bw_intra[g]), float(w.bw_inter[g]))):
            for k, v in enumerate(volumes):
                vol[g, link, k] = v
                if v == 0.0 or not np.isfinite(bw):
                    lat[g, link, k] = alpha[link] if np.isfinite(bw) else 0.0
                else:
                    lat[g, link, k] = alpha[link] + (v + half[link]) / bw
    return vol, lat


def linear_tables(w, K: int = 2):
    """Tables that reproduce volume / bandwidth: points (0, 0) and (bw, 1 s), and
    K - 2 more on the same line."""
    T = int(w.n_types)
    vol = np.zeros((T, 2, K), np.float64)
    lat = np.zeros((T, 2, K), np.float64)
    for g in range(T):
        for link, bw in enumerate((float(w.bw_intra[g]), float(w.bw_inter[g]))):
            for k in range(K):
                if np.isfinite(bw):
                    vol[g, link, k] = bw * k / (K - 1)
                    lat[g, link, k] = k / (K - 1)
                else:                      # a free link: no latency at any volume
                    vol[g, link, k] = float(k)
    return vol, lat
