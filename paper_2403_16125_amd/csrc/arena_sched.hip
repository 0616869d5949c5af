// HIP kernel of one scheduling step over the throughput matrix (gfx950).
//
// Event-driven scheduling with the throughput objective (Sec. 3.5,
// Algorithm 1, Eq. 5): queued jobs launch on the fastest grid that fits,
// cheapest scale-downs of running jobs (throughput lost per GPU freed) make
// room within the search depth, and the best scale-ups (throughput gained
// per GPU) use what is left.  The step is a chain of dependent decisions,
// each an arg-min over every job or grid, so one workgroup of 1024 threads
// runs the whole step: each decision is a block-wide reduction of
// (key, index) pairs -- index breaking ties -- over per-thread candidates.
// Costs and gains are float64 from the float32 matrix, in the same
// operation order as a plain evaluation, so every decision is reproducible.
#include <math.h>

#include "arena_internal.h"

namespace arena {
namespace {

constexpr int kSchedThreads = 1024;
constexpr int kSchedWaves = kSchedThreads / 64;
constexpr double kInfD = __builtin_huge_val();

struct Best {
    double key;     // smaller wins
    int idx;        // then the smaller index
    int aux;        // payload (a count index)
};

__device__ __forceinline__ bool better(const Best& a, const Best& b)
{
    return a.key < b.key || (a.key == b.key && a.idx < b.idx);
}

struct SchedLds {
    int32_t counts[kMaxSchedCounts];
    int32_t free[kMaxSchedTypes];
    double rkey[kSchedWaves];
    int32_t ridx[kSchedWaves];
    int32_t raux[kSchedWaves];
    int32_t log_job[kMaxSchedDepth];
    int32_t log_cnt[kMaxSchedDepth];
    unsigned long long usable;      // types where the queued job has a grid with throughput > 0
    int32_t bad;
    uint32_t queued_bits[kMaxSchedJobs / 32];
};

// Block-wide minimum of `b` (every thread receives the winner).
__device__ Best block_min(Best b, SchedLds& S)
{
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        Best o;
        o.key = __shfl_xor(b.key, off);
        o.idx = __shfl_xor(b.idx, off);
        o.aux = __shfl_xor(b.aux, off);
        if (better(o, b)) b = o;
    }
    if (lane == 0) {
        S.rkey[w] = b.key;
        S.ridx[w] = b.idx;
        S.raux[w] = b.aux;
    }
    __syncthreads();
    Best r{kInfD, 0x7fffffff, -1};
    for (int k = 0; k < kSchedWaves; ++k) {
        const Best o{S.rkey[k], S.ridx[k], S.raux[k]};
        if (better(o, r)) r = o;
    }
    __syncthreads();
    return r;
}

// S2: the fastest grid of job j that fits the free GPUs (key -thr, index c*64+g).
__device__ Best launch_grid(const SchedArgs& A, SchedLds& S, int j)
{
    Best b{kInfD, 0x7fffffff, -1};
    const float* row = A.thr + (size_t)j * A.n_types * A.n_counts;
    for (int e = threadIdx.x; e < A.n_types * A.n_counts; e += kSchedThreads) {
        const int g = e / A.n_counts, c = e - g * A.n_counts;
        const float v = row[e];
        if (v > 0.0f && S.counts[c] <= S.free[g]) {
            const Best o{-(double)v, c * 64 + g, e};
            if (better(o, b)) b = o;
        }
    }
    return block_min(b, S);
}

// S3: the cheapest scale-down on a type the queued job can use.
__device__ Best scale_down(const SchedArgs& A, SchedLds& S)
{
    Best b{kInfD, 0x7fffffff, -1};
    for (int i = threadIdx.x; i < A.n_jobs; i += kSchedThreads) {
        const int g = A.alloc_type[i];
        if (g < 0 || !((S.usable >> g) & 1ull)) continue;
        const int c = A.alloc_count[i];
        const float* row = A.thr + ((size_t)i * A.n_types + g) * A.n_counts;
        int c2 = c - 1;
        while (c2 >= 0 && !(row[c2] > 0.0f)) --c2;
        if (c2 < 0) continue;
        const double cost = ((double)row[c] - (double)row[c2]) / (double)(S.counts[c] - S.counts[c2]);
        const Best o{cost, i, c2};
        if (better(o, b)) b = o;
    }
    return block_min(b, S);
}

// S6: the scale-up with the largest gain per GPU (key -gain).
__device__ Best scale_up(const SchedArgs& A, SchedLds& S)
{
    Best b{kInfD, 0x7fffffff, -1};
    for (int i = threadIdx.x; i < A.n_jobs; i += kSchedThreads) {
        const int g = A.alloc_type[i];
        if (g < 0) continue;
        const int c = A.alloc_count[i];
        const float* row = A.thr + ((size_t)i * A.n_types + g) * A.n_counts;
        const int n = S.counts[c];
        const double t = (double)row[c];
        double gbest = -kInfD;
        int cbest = -1;
        for (int c2 = c + 1; c2 < A.n_counts; ++c2) {
            const int dn = S.counts[c2] - n;
            if (dn > S.free[g]) break;
            const double t2 = (double)row[c2];
            if (t2 > t) {
                const double gain = (t2 - t) / (double)dn;
                if (gain > gbest) {
                    gbest = gain;
                    cbest = c2;
                }
            }
        }
        if (cbest < 0) continue;
        const Best o{-gbest, i, cbest};
        if (better(o, b)) b = o;
    }
    return block_min(b, S);
}

__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(SchedArgs A)
{
    __shared__ SchedLds S;
    const int tid = threadIdx.x;
    for (int c = tid; c < A.n_counts; c += kSchedThreads) S.counts[c] = A.counts[c];
    for (int g = tid; g < A.n_types; g += kSchedThreads) S.free[g] = A.capacity[g];
    for (int k = tid; k < (A.n_jobs + 31) / 32; k += kSchedThreads) S.queued_bits[k] = 0u;
    if (tid == 0) S.bad = 0;
    __syncthreads();
    // occupied GPUs; every index in range; queued jobs distinct and not running
    for (int i = tid; i < A.n_jobs; i += kSchedThreads) {
        const int g = A.alloc_type[i], c = A.alloc_count[i];
        if (g >= 0) {
            if (g >= A.n_types || c < 0 || c >= A.n_counts) atomicOr(&S.bad, 2);
            else atomicSub(&S.free[g], S.counts[c]);
        }
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

    int kept_down = 0, launches = 0, ups = 0;
    int lam = 0;
    for (int q = 0; q < A.n_queue; ++q) lam = max(lam, A.priority[q]);
    lam += 1;

    for (int q = 0; q < A.n_queue; ++q) {
        const int j = A.queue[q];
        // S3: types where job j has a grid with throughput > 0
        if (tid == 0) S.usable = 0ull;
        __syncthreads();
        const float* row = A.thr + (size_t)j * A.n_types * A.n_counts;
        for (int e = tid; e < A.n_types * A.n_counts; e += kSchedThreads)
            if (row[e] > 0.0f) atomicOr(&S.usable, 1ull << (e / A.n_counts));
        __syncthreads();
        int nlog = 0;
        bool ok = false;
        for (;;) {
            const Best lg = launch_grid(A, S, j);
            if (lg.aux >= 0) {
                const int g = lg.aux / A.n_counts, c = lg.aux - g * A.n_counts;
                if (tid == 0) {
                    A.alloc_type[j] = g;
                    A.alloc_count[j] = c;
                    S.free[g] -= S.counts[c];
                }
                ok = true;
                break;
            }
            if (nlog >= A.depth) break;
            const Best sd = scale_down(A, S);
            if (sd.aux < 0) break;
            if (tid == 0) {
                const int i = sd.idx, g = A.alloc_type[i];
                S.log_job[nlog] = i;
                S.log_cnt[nlog] = A.alloc_count[i];
                S.free[g] += S.counts[A.alloc_count[i]] - S.counts[sd.aux];
                A.alloc_count[i] = sd.aux;
            }
            ++nlog;
            __syncthreads();
        }
        if (ok) {
            ++launches;
            kept_down += nlog;
        } else if (tid == 0) {
            // S4: undo, newest first
            for (int k = nlog - 1; k >= 0; --k) {
                const int i = S.log_job[k], g = A.alloc_type[i];
                S.free[g] -= S.counts[S.log_cnt[k]] - S.counts[A.alloc_count[i]];
                A.alloc_count[i] = S.log_cnt[k];
            }
        }
        if (tid == 0) A.launched[q] = ok ? 1 : 0;
        __syncthreads();
        if (!ok) {                       // S5
            if (A.priority[q] <= lam) lam = A.priority[q];
            else break;
        }
    }
    while (ups < A.depth) {              // S6
        const Best su = scale_up(A, S);
        if (su.aux < 0) break;
        if (tid == 0) {
            const int i = su.idx, g = A.alloc_type[i];
            S.free[g] -= S.counts[su.aux] - S.counts[A.alloc_count[i]];
            A.alloc_count[i] = su.aux;
        }
        ++ups;
        __syncthreads();
    }
    if (tid == 0) {
        A.result[0] = 0;
        A.result[1] = kept_down;
        A.result[2] = launches;
        A.result[3] = ups;
    }
}

}  // namespace

hipError_t launch_schedule(const SchedArgs& args, hipStream_t stream)
{
    hipLaunchKernelGGL(schedule_kernel, dim3(1), dim3(kSchedThreads), 0, stream, args);
    return hipGetLastError();
}

}  // namespace arena
