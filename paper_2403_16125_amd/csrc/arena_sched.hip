// HIP kernel of one scheduling step over the throughput matrix (gfx950).
//
// Event-driven scheduling with the throughput objective (Sec. 3.5,
// Algorithm 1, Eq. 5): queued jobs launch on the fastest grid that fits,
// cheapest scale-downs of running jobs (throughput lost per GPU freed) make
// room within the search depth, and the best scale-ups (throughput gained
// per GPU) use what is left.  Under the finish-time fairness objective
// (Eq. 7) the two searches rank by rho = B N / (thr n) instead: the job
// whose rho after its scale-down is least, and the worst-off job moved to
// its least-rho count.  The step is a chain of dependent decisions,
// each an arg-min over the running jobs or over one job's grids, so one
// workgroup runs the whole step and each decision is a block-wide reduction
// of (key, index) pairs -- index breaking ties -- over per-thread candidates.
//
// The step is latency-bound (one small decision after another), so the
// design removes latency from each decision:
//  * the running jobs are compacted into an LDS list at the start, with each
//    one's allocation and best scale-down (cost, count, type) cached beside
//    it: a move changes one job, so only its entry is recomputed, and a
//    scale-down search is one pass over LDS;
//  * the next queued job's throughput row is loaded while the current job is
//    visited (all loads of a thread in flight together) and staged in LDS,
//    so every launch decision reads LDS;
//  * a decision reduces within each wave by DPP row rotations (VALU, no LDS
//    traffic) and read-lanes, and across the 4 waves through a double-
//    buffered LDS slot: one barrier per decision.
// When more jobs run than the list holds, the step scans every job instead
// (same decisions, slower).  Costs and gains are float64 from the float32
// matrix, in the same operation order as a plain evaluation, so every
// decision is reproducible.
#include <math.h>

#include "arena_internal.h"

namespace arena {
namespace {

constexpr int kSchedThreads = 256;
constexpr int kSchedWaves = kSchedThreads / 64;
constexpr int kMaxRun = 4096;            // running jobs tracked in LDS
constexpr int kRowUnroll = 8;            // row loads a thread keeps in flight
constexpr int kRowBuf = kRowUnroll * kSchedThreads;  // grids of a row staged in LDS
constexpr double kInfD = __builtin_huge_val();
constexpr int kNone = 0x7fffffff;

struct Best {
    double key;     // smaller wins
    int idx;        // then the smaller index
    int aux;        // payload (a count index or a grid)
    int slot;       // payload (the job's slot in the running list)
};

__device__ __forceinline__ bool better(double ka, int ia, double kb, int ib)
{
    return ka < kb || (ka == kb && ia < ib);
}

struct SchedLds {
    int32_t counts[kMaxSchedCounts];
    int32_t free[kMaxSchedTypes];
    // cross-wave reduction slots, double-buffered
    double rkey[2][kSchedWaves];
    int32_t ridx[2][kSchedWaves];
    int32_t raux[2][kSchedWaves];
    int32_t rslot[2][kSchedWaves];
    unsigned long long rmask[2][kSchedWaves];
    unsigned long long rk64[2][kSchedWaves];
    int32_t log_job[kMaxSchedDepth];
    int32_t log_cnt[kMaxSchedDepth];
    int32_t log_slot[kMaxSchedDepth];
    double log_cost[kMaxSchedDepth];
    int32_t log_info[kMaxSchedDepth];
    unsigned long long usable;      // types where the queued job has an open grid
    int32_t bad;
    int32_t pmax;                   // largest priority class in the queue
    int32_t n_run;                  // running jobs in the list
    int32_t use_list;               // 0: more jobs run than the list holds, scan all jobs
    int32_t run[kMaxRun];           // running job ids (any order)
    int32_t ralloc[kMaxRun];        // their count index | type << 16
    double dcost[kMaxRun];          // cached best scale-down cost of run[k]
    int32_t dinfo[kMaxRun];         // its target count | type << 16, -1 if it has none
    uint32_t queued_bits[kMaxSchedJobs / 32];
    float row[2][kRowBuf];          // visited job's row and the next one's (when they fit)
};

// DPP row rotation (all 64 lanes active; a rotation has no invalid source).
template <int CTRL>
__device__ __forceinline__ int dpp(int v)
{
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, false);
}

template <int CTRL>
__device__ __forceinline__ double dpp(double v)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const unsigned lo = (unsigned)dpp<CTRL>((int)(unsigned)u);
    const unsigned hi = (unsigned)dpp<CTRL>((int)(unsigned)(u >> 32));
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

template <int CTRL>
__device__ __forceinline__ void rot_min(double& k, int& i)
{
    const double ko = dpp<CTRL>(k);
    const int io = dpp<CTRL>(i);
    if (better(ko, io, k, i)) {
        k = ko;
        i = io;
    }
}

__device__ __forceinline__ double readlane_d(double v, int lane)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(v);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, lane);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), lane);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Block-wide arg-min of (key, idx) with its payload (every thread receives
// the result).  Rotations within each 16-lane row, read-lanes across the 4
// rows, then the 4 waves through LDS slot `phase` (alternating, so no
// barrier is needed after the read).
__device__ __forceinline__ Best block_min(const Best& b, SchedLds& S, int& phase)
{
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    double k = b.key;
    int i = b.idx;
    rot_min<0x121>(k, i);
    rot_min<0x122>(k, i);
    rot_min<0x124>(k, i);
    rot_min<0x128>(k, i);
    double K = readlane_d(k, 0);
    int I = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
    for (int r = 1; r < 4; ++r) {
        const double kr = readlane_d(k, 16 * r);
        const int ir = __builtin_amdgcn_readlane(i, 16 * r);
        if (better(kr, ir, K, I)) {
            K = kr;
            I = ir;
        }
    }
    // the winning lane (candidates are distinct; lanes without one all hold
    // (inf, kNone) and any of them will do)
    const unsigned long long win = __ballot(b.key == K && b.idx == I);
    const int wl = win ? __ffsll((long long)win) - 1 : 0;
    const int aux = __builtin_amdgcn_readlane(b.aux, wl);
    const int slot = __builtin_amdgcn_readlane(b.slot, wl);
    const int ph = phase;
    phase ^= 1;
    if (lane == 0) {
        S.rkey[ph][w] = K;
        S.ridx[ph][w] = I;
        S.raux[ph][w] = aux;
        S.rslot[ph][w] = slot;
    }
    __syncthreads();
    Best r{S.rkey[ph][0], S.ridx[ph][0], S.raux[ph][0], S.rslot[ph][0]};
#pragma unroll
    for (int q = 1; q < kSchedWaves; ++q) {
        const double kq = S.rkey[ph][q];
        const int iq = S.ridx[ph][q];
        if (better(kq, iq, r.key, r.idx)) r = Best{kq, iq, S.raux[ph][q], S.rslot[ph][q]};
    }
    return r;
}

// Launch candidates pack into one unsigned 64-bit order: higher throughput
// first (v > 0, finite or +inf, so ~bits & 0x7fffffff falls as v grows), then
// the smaller count index, then the lower type.
__device__ __forceinline__ unsigned long long launch_key(float v, int c, int g)
{
    const unsigned hi = ~__float_as_uint(v) & 0x7fffffffu;
    return ((unsigned long long)hi << 32) | (unsigned)(c * 64 + g);
}

template <int CTRL>
__device__ __forceinline__ unsigned long long dpp64(unsigned long long v)
{
    const unsigned lo = (unsigned)dpp<CTRL>((int)(unsigned)v);
    const unsigned hi = (unsigned)dpp<CTRL>((int)(unsigned)(v >> 32));
    return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ unsigned long long readlane64(unsigned long long v, int lane)
{
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)v, lane);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(v >> 32), lane);
    return ((unsigned long long)hi << 32) | lo;
}

// Block-wide minimum of a packed key and, when asked, OR of `mask`.
__device__ __forceinline__ unsigned long long block_min64(unsigned long long k, SchedLds& S, int& phase,
                                                          bool want_mask, unsigned long long& mask)
{
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    unsigned long long o;
    o = dpp64<0x121>(k); k = o < k ? o : k;
    o = dpp64<0x122>(k); k = o < k ? o : k;
    o = dpp64<0x124>(k); k = o < k ? o : k;
    o = dpp64<0x128>(k); k = o < k ? o : k;
    unsigned long long K = readlane64(k, 0);
#pragma unroll
    for (int r = 1; r < 4; ++r) {
        const unsigned long long kr = readlane64(k, 16 * r);
        K = kr < K ? kr : K;
    }
    unsigned long long M = 0ull;
    if (want_mask) {
        unsigned long long m = mask;
        m |= dpp64<0x121>(m);
        m |= dpp64<0x122>(m);
        m |= dpp64<0x124>(m);
        m |= dpp64<0x128>(m);
#pragma unroll
        for (int r = 0; r < 4; ++r) M |= readlane64(m, 16 * r);
    }
    const int ph = phase;
    phase ^= 1;
    if (lane == 0) {
        S.rk64[ph][w] = K;
        S.rmask[ph][w] = M;
    }
    __syncthreads();
    unsigned long long r = S.rk64[ph][0], mr = S.rmask[ph][0];
#pragma unroll
    for (int q = 1; q < kSchedWaves; ++q) {
        const unsigned long long kq = S.rk64[ph][q];
        r = kq < r ? kq : r;
        mr |= S.rmask[ph][q];
    }
    if (want_mask) mask = mr;
    return r;
}

// Work of job i to finish (batch x remaining iterations, when the deadline
// constraint or the fairness objective needs it) and its deadline; dl < 0
// when there is no deadline constraint.
template <bool DDL, bool FAIR = false>
__device__ __forceinline__ void job_deadline(const SchedArgs& A, int i, double& bn, double& dl)
{
    bn = (DDL || FAIR) ? (double)A.batch[i] * (double)A.iters[i] : 0.0;
    dl = DDL ? (double)A.ddl[i] : -1.0;
}

// Finish-time-fairness ratio (Eq. 7) of a job with work bn at throughput v
// on n GPUs: the remaining time bn / v per GPU; +inf at v = 0.
__device__ __forceinline__ double fair_rho(float v, int n, double bn)
{
    return v > 0.0f ? bn / ((double)v * (double)n) : kInfD;
}

// A grid of throughput v is open to the job: v > 0 and, under the deadline
// constraint (Eq. 6), the remaining work finishes in time at v.
template <bool DDL>
__device__ __forceinline__ bool open_grid(float v, double bn, double dl)
{
    if (!DDL) return v > 0.0f;
    return v > 0.0f && bn / (double)v <= dl;
}

// S2: the fastest grid of job j that fits the free GPUs (payload the grid
// index g*NC + c, -1 if none fits), and on the first pass of a visit the
// types where j has an open grid.  A staged row is read from
// LDS buffer `buf` with each thread's grids (type, count index, GPU count)
// decoded once in `eg`; a larger row is read from memory and decoded here.
template <bool DDL>
__device__ __forceinline__ Best launch_grid(const SchedArgs& A, SchedLds& S, int j, int buf, bool first, int& phase,
                            unsigned long long& usable, const int (&eg)[kRowUnroll])
{
    unsigned long long best = ~0ull, m = 0ull;
    double bn, dl;
    job_deadline<DDL>(A, j, bn, dl);
    const int nc = A.n_counts, ng = A.n_types * nc;
    if (ng <= kRowBuf) {
        float v[kRowUnroll];
        int fr[kRowUnroll];
#pragma unroll
        for (int u = 0; u < kRowUnroll; ++u) {
            v[u] = eg[u] >= 0 ? S.row[buf][threadIdx.x + u * kSchedThreads] : 0.0f;
            fr[u] = S.free[eg[u] & 63];
        }
#pragma unroll
        for (int u = 0; u < kRowUnroll; ++u) {
            if (eg[u] >= 0 && open_grid<DDL>(v[u], bn, dl)) {
                const int g = eg[u] & 63;
                m |= 1ull << g;
                if ((eg[u] >> 15) <= fr[u]) {
                    const unsigned long long k = launch_key(v[u], (eg[u] >> 6) & 511, g);
                    best = k < best ? k : best;
                }
            }
        }
    } else {
        const float* row = A.thr + (size_t)j * ng;
        for (int base = threadIdx.x; base < ng; base += kSchedThreads * kRowUnroll) {
            float v[kRowUnroll];
#pragma unroll
            for (int u = 0; u < kRowUnroll; ++u) {
                const int e = base + u * kSchedThreads;
                v[u] = e < ng ? row[e] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < kRowUnroll; ++u) {
                const int e = base + u * kSchedThreads;
                if (e < ng && open_grid<DDL>(v[u], bn, dl)) {
                    const int g = e / nc, c = e - g * nc;
                    m |= 1ull << g;
                    if (S.counts[c] <= S.free[g]) {
                        const unsigned long long k = launch_key(v[u], c, g);
                        best = k < best ? k : best;
                    }
                }
            }
        }
    }
    best = block_min64(best, S, phase, first, m);
    if (first) usable = m;
    Best r{0.0, 0, -1, -1};
    if (best != ~0ull) {
        const int idx = (int)(unsigned)best;
        r.aux = (idx & 63) * nc + (idx >> 6);
    }
    return r;
}

// S3 for one running job: the largest smaller count open to it and the
// throughput lost per GPU freed (under fairness: the job's rho there);
// c2 = -1 if there is none.
template <bool DDL, bool FAIR>
__device__ __forceinline__ double down_cost(const SchedArgs& A, const SchedLds& S, int i, int g, int c,
                                            int& c2)
{
    const float* row = A.thr + ((size_t)i * A.n_types + g) * A.n_counts;
    double bn, dl;
    job_deadline<DDL, FAIR>(A, i, bn, dl);
    const float tc = row[c];
    c2 = c - 1;
    float t2 = c2 >= 0 ? row[c2] : 0.0f;
    while (c2 >= 0 && !open_grid<DDL>(t2, bn, dl)) {
        --c2;
        t2 = c2 >= 0 ? row[c2] : 0.0f;
    }
    if (c2 < 0) return kInfD;
    if (FAIR) return fair_rho(t2, S.counts[c2], bn);
    const double cost = ((double)tc - (double)t2) / (double)(S.counts[c] - S.counts[c2]);
    if (cost != cost) c2 = -1;      // not a number (infinite throughputs): no candidate
    return cost;
}

// Refreshes the cached scale-down of list slot k from S.ralloc[k] (one thread).
template <bool DDL, bool FAIR>
__device__ __forceinline__ void cache_slot(const SchedArgs& A, SchedLds& S, int k)
{
    const int al = S.ralloc[k], g = al >> 16;
    int c2;
    const double cost = down_cost<DDL, FAIR>(A, S, S.run[k], g, al & 0xffff, c2);
    S.dcost[k] = cost;
    S.dinfo[k] = c2 < 0 ? -1 : (c2 | (g << 16));
}

// S3: the cheapest scale-down on a type the queued job can use.
template <bool DDL, bool FAIR>
__device__ Best scale_down(const SchedArgs& A, SchedLds& S, int& phase)
{
    Best b{kInfD, kNone, -1, -1};
    const unsigned long long usable = S.usable;
    if (S.use_list) {
        for (int k = threadIdx.x; k < S.n_run; k += kSchedThreads) {
            const int info = S.dinfo[k];
            if (info < 0 || !((usable >> (info >> 16)) & 1ull)) continue;
            const double key = S.dcost[k];
            const int idx = S.run[k];
            if (better(key, idx, b.key, b.idx)) b = Best{key, idx, info & 0xffff, k};
        }
    } else {
        for (int i = threadIdx.x; i < A.n_jobs; i += kSchedThreads) {
            const int g = A.alloc_type[i];
            if (g < 0 || !((usable >> g) & 1ull)) continue;
            int c2;
            const double cost = down_cost<DDL, FAIR>(A, S, i, g, A.alloc_count[i], c2);
            if (c2 < 0) continue;
            if (better(cost, i, b.key, b.idx)) b = Best{cost, i, c2, -1};
        }
    }
    return block_min(b, S, phase);
}

// S6 for one running job (type g, count index c): its best scale-up within
// the free GPUs (gain per added GPU; ties to the smaller count).  Under
// fairness: the count with the least rho, a candidate only if that is below
// the current rho, keyed by -(current rho) so the worst-off job wins.
template <bool DDL, bool FAIR>
__device__ __forceinline__ void up_move(const SchedArgs& A, const SchedLds& S, int i, int g, int c, int k,
                                        Best& b)
{
    const float* row = A.thr + ((size_t)i * A.n_types + g) * A.n_counts;
    double bn, dl;
    job_deadline<DDL, FAIR>(A, i, bn, dl);
    const int n = S.counts[c];
    const int fr = S.free[g];
    if (FAIR) {
        const double r0 = fair_rho(row[c], n, bn);
        double rbest = kInfD;
        int cb = -1;
        for (int c2 = c + 1; c2 < A.n_counts; ++c2) {
            const int n2 = S.counts[c2];
            if (n2 - n > fr) break;
            const float v2 = row[c2];
            if (open_grid<DDL>(v2, bn, dl)) {
                const double r2 = fair_rho(v2, n2, bn);
                if (cb < 0 || r2 < rbest) {
                    rbest = r2;
                    cb = c2;
                }
            }
        }
        if (cb >= 0 && rbest < r0 && better(-r0, i, b.key, b.idx)) b = Best{-r0, i, cb, k};
        return;
    }
    const double t = (double)row[c];
    double gbest = -kInfD;
    int cbest = -1;
    for (int c2 = c + 1; c2 < A.n_counts; ++c2) {
        const int dn = S.counts[c2] - n;
        if (dn > fr) break;
        const float v2 = row[c2];
        const double t2 = (double)v2;
        if (t2 > t && open_grid<DDL>(v2, bn, dl)) {
            const double gain = (t2 - t) / (double)dn;
            if (gain > gbest) {
                gbest = gain;
                cbest = c2;
            }
        }
    }
    if (cbest < 0) return;
    if (better(-gbest, i, b.key, b.idx)) b = Best{-gbest, i, cbest, k};
}

// S6: the scale-up with the largest gain per GPU (key -gain).
template <bool DDL, bool FAIR>
__device__ Best scale_up(const SchedArgs& A, SchedLds& S, int& phase)
{
    Best b{kInfD, kNone, -1, -1};
    if (S.use_list) {
        for (int k = threadIdx.x; k < S.n_run; k += kSchedThreads) {
            const int al = S.ralloc[k];
            up_move<DDL, FAIR>(A, S, S.run[k], al >> 16, al & 0xffff, k, b);
        }
    } else {
        for (int i = threadIdx.x; i < A.n_jobs; i += kSchedThreads) {
            const int g = A.alloc_type[i];
            if (g >= 0) up_move<DDL, FAIR>(A, S, i, g, A.alloc_count[i], -1, b);
        }
    }
    return block_min(b, S, phase);
}

template <bool DDL, bool FAIR>
__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(SchedArgs A)
{
    __shared__ SchedLds S;
    const int tid = threadIdx.x;
    for (int c = tid; c < A.n_counts; c += kSchedThreads) S.counts[c] = A.counts[c];
    for (int g = tid; g < A.n_types; g += kSchedThreads) S.free[g] = A.capacity[g];
    for (int k = tid; k < (A.n_jobs + 31) / 32; k += kSchedThreads) S.queued_bits[k] = 0u;
    if (tid == 0) {
        S.bad = 0;
        S.pmax = 0;
        S.n_run = 0;
    }
    __syncthreads();
    // occupied GPUs and the running list; every index in range; queued jobs
    // distinct and not running
    for (int i = tid; i < A.n_jobs; i += kSchedThreads) {
        const int g = A.alloc_type[i], c = A.alloc_count[i];
        if (g >= 0) {
            if (g >= A.n_types || c < 0 || c >= A.n_counts) {
                atomicOr(&S.bad, 2);
            } else {
                atomicSub(&S.free[g], S.counts[c]);
                const int k = atomicAdd(&S.n_run, 1);
                if (k < kMaxRun) {
                    S.run[k] = i;
                    S.ralloc[k] = c | (g << 16);
                }
            }
        }
    }
    if (DDL || FAIR)
        for (int i = tid; i < A.n_jobs; i += kSchedThreads) {
            const float it = A.iters[i];
            if (A.batch[i] <= 0 || !(it >= 0.0f) || it == __builtin_huge_valf() || (DDL && !(A.ddl[i] > 0.0f)))
                atomicOr(&S.bad, 2);
        }
    for (int q = tid; q < A.n_queue; q += kSchedThreads) {
        const int j = A.queue[q];
        if (j < 0 || j >= A.n_jobs || A.alloc_type[j] >= 0 || A.priority[q] < 0) {
            atomicOr(&S.bad, 2);
        } else {
            const uint32_t bit = 1u << (j & 31);
            if (atomicOr(&S.queued_bits[j >> 5], bit) & bit) atomicOr(&S.bad, 2);
        }
    }
    __syncthreads();
    for (int g = tid; g < A.n_types; g += kSchedThreads)
        if (S.free[g] < 0) atomicOr(&S.bad, 1);
    __syncthreads();
    if (S.bad) {
        if (tid == 0) A.result[0] = (S.bad & 2) ? 2 : 1;
        return;
    }
    // jobs the visit does not reach stay queued
    for (int q = tid; q < A.n_queue; q += kSchedThreads) A.launched[q] = 0;
    const bool fits = S.n_run <= kMaxRun;
    if (fits)
        for (int k = tid; k < S.n_run; k += kSchedThreads) cache_slot<DDL, FAIR>(A, S, k);
    __syncthreads();
    if (tid == 0) S.use_list = fits ? 1 : 0;
    __syncthreads();

    int phase = 0;
    int kept_down = 0, launches = 0, ups = 0;
    int passes = 0;                  // decisions taken (launch, scale-down and scale-up searches)
    unsigned long long scanned = 0;  // candidates those searches examined
    // S5: lam' starts above every class
    {
        int pm = 0;
        for (int q = tid; q < A.n_queue; q += kSchedThreads) pm = max(pm, A.priority[q]);
        atomicMax(&S.pmax, pm);
    }
    __syncthreads();
    int lam = S.pmax + 1;

    // rows of queued jobs are staged in LDS (double-buffered) when they fit;
    // each thread then always handles the grids tid + u * threads, decoded
    // once: type | count index << 6 | GPU count << 15, -1 past the row
    const int ng = A.n_types * A.n_counts;
    const bool staged = ng <= kRowBuf;
    int eg[kRowUnroll];
#pragma unroll
    for (int u = 0; u < kRowUnroll; ++u) {
        const int e = tid + u * kSchedThreads;
        if (staged && e < ng) {
            const int g = e / A.n_counts, c = e - g * A.n_counts;
            eg[u] = g | (c << 6) | (S.counts[c] << 15);
        } else {
            eg[u] = -1;
        }
    }
    if (staged && A.n_queue > 0) {
        const float* row0 = A.thr + (size_t)A.queue[0] * ng;
        for (int e = tid; e < ng; e += kSchedThreads) S.row[0][e] = row0[e];
    }
    __syncthreads();

    for (int q = 0; q < A.n_queue; ++q) {
        const int j = A.queue[q];
        const int buf = q & 1;
        // the next job's row: loads issued now, staged at the end of the visit
        const bool pf = staged && q + 1 < A.n_queue;
        float next[kRowUnroll];
        if (pf) {
            const float* nrow = A.thr + (size_t)A.queue[q + 1] * ng;
#pragma unroll
            for (int u = 0; u < kRowUnroll; ++u) {
                const int e = tid + u * kSchedThreads;
                next[u] = e < ng ? nrow[e] : 0.0f;
            }
        }
        int nlog = 0;
        bool ok = false;
        for (;;) {
            unsigned long long usable = 0ull;
            const Best lg = launch_grid<DDL>(A, S, j, buf, nlog == 0, phase, usable, eg);
            ++passes;
            scanned += (unsigned long long)ng;
            if (lg.aux >= 0) {
                const int g = lg.aux / A.n_counts, c = lg.aux - g * A.n_counts;
                if (tid == 0) {
                    A.alloc_type[j] = g;
                    A.alloc_count[j] = c;
                    S.free[g] -= S.counts[c];
                    if (S.use_list) {
                        if (S.n_run < kMaxRun) {
                            const int k = S.n_run++;
                            S.run[k] = j;
                            S.ralloc[k] = c | (g << 16);
                            cache_slot<DDL, FAIR>(A, S, k);
                        } else {
                            S.use_list = 0;
                        }
                    }
                }
                ok = true;
                break;
            }
            if (nlog >= A.depth) break;
            if (nlog == 0 && tid == 0) S.usable = usable;
            __syncthreads();
            ++passes;
            scanned += (unsigned long long)(S.use_list ? S.n_run : A.n_jobs);
            const Best sd = scale_down<DDL, FAIR>(A, S, phase);
            if (sd.aux < 0) break;
            if (tid == 0) {
                const int i = sd.idx;
                int g, c;
                if (sd.slot >= 0) {
                    const int al = S.ralloc[sd.slot];
                    g = al >> 16;
                    c = al & 0xffff;
                } else {
                    g = A.alloc_type[i];
                    c = A.alloc_count[i];
                }
                S.log_job[nlog] = i;
                S.log_cnt[nlog] = c;
                S.log_slot[nlog] = sd.slot;
                S.free[g] += S.counts[c] - S.counts[sd.aux];
                A.alloc_count[i] = sd.aux;
                if (sd.slot >= 0) {
                    S.log_cost[nlog] = S.dcost[sd.slot];
                    S.log_info[nlog] = S.dinfo[sd.slot];
                    S.ralloc[sd.slot] = sd.aux | (g << 16);
                    cache_slot<DDL, FAIR>(A, S, sd.slot);
                }
            }
            ++nlog;
            __syncthreads();
        }
        if (ok) {
            ++launches;
            kept_down += nlog;
        } else if (tid == 0) {
            // S4: undo, newest first (cached entries restored with them)
            for (int k = nlog - 1; k >= 0; --k) {
                const int i = S.log_job[k], slot = S.log_slot[k];
                int g, cnow;
                if (slot >= 0) {
                    const int al = S.ralloc[slot];
                    g = al >> 16;
                    cnow = al & 0xffff;
                    S.ralloc[slot] = S.log_cnt[k] | (g << 16);
                    S.dcost[slot] = S.log_cost[k];
                    S.dinfo[slot] = S.log_info[k];
                } else {
                    g = A.alloc_type[i];
                    cnow = A.alloc_count[i];
                }
                S.free[g] -= S.counts[S.log_cnt[k]] - S.counts[cnow];
                A.alloc_count[i] = S.log_cnt[k];
            }
        }
        if (pf) {
#pragma unroll
            for (int u = 0; u < kRowUnroll; ++u) {
                const int e = tid + u * kSchedThreads;
                if (e < ng) S.row[buf ^ 1][e] = next[u];
            }
        }
        if (tid == 0) A.launched[q] = ok ? 1 : 0;
        __syncthreads();
        if (!ok) {                       // S5
            const int pq = A.priority[q];
            if (pq <= lam) lam = pq;
            else break;
        }
    }
    while (ups < A.depth) {              // S6
        ++passes;
        scanned += (unsigned long long)(S.use_list ? S.n_run : A.n_jobs);
        const Best su = scale_up<DDL, FAIR>(A, S, phase);
        if (su.aux < 0) break;
        if (tid == 0) {
            const int i = su.idx;
            int g, c;
            if (su.slot >= 0) {
                const int al = S.ralloc[su.slot];
                g = al >> 16;
                c = al & 0xffff;
            } else {
                g = A.alloc_type[i];
                c = A.alloc_count[i];
            }
            S.free[g] -= S.counts[su.aux] - S.counts[c];
            A.alloc_count[i] = su.aux;
            if (su.slot >= 0) {
                S.ralloc[su.slot] = su.aux | (g << 16);
                cache_slot<DDL, FAIR>(A, S, su.slot);
            }
        }
        ++ups;
        __syncthreads();
    }
    if (tid == 0) {
        A.result[0] = 0;
        A.result[1] = kept_down;
        A.result[2] = launches;
        A.result[3] = ups;
        A.result[4] = passes;
        A.result[5] = (int32_t)(uint32_t)scanned;
        A.result[6] = (int32_t)(uint32_t)(scanned >> 32);
        A.result[7] = 0;
    }
}

}  // namespace

hipError_t launch_schedule(const SchedArgs& args, hipStream_t stream)
{
    const dim3 grid(1), block(kSchedThreads);
    if (args.objective == 1) {
        if (args.ddl) hipLaunchKernelGGL((schedule_kernel<true, true>), grid, block, 0, stream, args);
        else hipLaunchKernelGGL((schedule_kernel<false, true>), grid, block, 0, stream, args);
    } else {
        if (args.ddl) hipLaunchKernelGGL((schedule_kernel<true, false>), grid, block, 0, stream, args);
        else hipLaunchKernelGGL((schedule_kernel<false, false>), grid, block, 0, stream, args);
    }
    return hipGetLastError();
}

}  // namespace arena
