// HIP kernels of the plan-space estimator (gfx950 / CDNA4).
//
// One 64-lane wavefront owns one (job, GPU type) pair and walks the GPU counts
// of the grid.  For each count it solves the stage-partition problems of the
// cell (one per tensor degree, plus the no-all-to-all variant of MoE jobs),
// prices every plan, and reduces to the cell's best plan.  Nothing here is a
// dense contraction, so no MFMA: the work is compares, min/max and adds on
// the vector ALU, with the job's tables, the prefix sums and the recursion
// rows staged in LDS.
//
// Arithmetic is IEEE double.  The per-layer cost, its prefix sums, the
// balanced-partition value and the canonical cuts are evaluated in the same
// operation order as a plain left-to-right evaluation of the formulas in
// arena.h, so they are bit-reproducible; only the sum of stage times is
// reduced in tree order.
#include <math.h>

#include "arena_internal.h"

namespace arena {
namespace {

constexpr double kInf = __builtin_huge_val();

struct Lds {
    double U[kLmax + 1];        // prefix of the per-sample layer cost of the current problem
    double Pp[kLmax + 1];       // prefix of parameter bytes of the job
    double Ap[kLmax + 1];       // prefix of activation bytes of the job
    double D[2][kLmax + 1];     // two rows of the partition recursion
    double planT[kMaxPlans];    // iteration time of each plan of the cell (+inf: does not fit)
    double planW[kMaxPlans];    // its slowest stage per sample
    uint32_t planKey[kMaxPlans];
    float t[kLmax];
    float x[kLmax];
    float q[kLmax];
    int32_t tg[kMaxTargets];    // pipeline degrees requested of the current problem, ascending
};

__device__ __forceinline__ void sync() { __syncthreads(); }

__device__ __forceinline__ double bcast(double v, int src)
{
    unsigned long long b = (unsigned long long)__double_as_longlong(v);
    int lo = __builtin_amdgcn_readlane((int)(unsigned)(b & 0xffffffffull), src);
    int hi = __builtin_amdgcn_readlane((int)(unsigned)(b >> 32), src);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) |
                                            (unsigned long long)(unsigned)lo));
}

__device__ __forceinline__ double wave_max(double v)
{
    for (int m = 32; m >= 1; m >>= 1) v = fmax(v, __shfl_xor(v, m));
    return v;
}

__device__ __forceinline__ double wave_min(double v)
{
    for (int m = 32; m >= 1; m >>= 1) v = fmin(v, __shfl_xor(v, m));
    return v;
}

// Tree sum; every lane returns lane 0's value so the result is uniform.
__device__ __forceinline__ double wave_sum(double v)
{
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return bcast(v, 0);
}

__device__ __forceinline__ unsigned wave_min_u(unsigned v)
{
    for (int m = 32; m >= 1; m >>= 1) {
        unsigned o = (unsigned)__shfl_xor((int)v, m);
        v = o < v ? o : v;
    }
    return v;
}

__device__ __forceinline__ int wave_max_i(int v)
{
    for (int m = 32; m >= 1; m >>= 1) {
        int o = __shfl_xor(v, m);
        v = o > v ? o : v;
    }
    return v;
}

// Left-to-right prefix sum of a per-lane pair (element lane, element lane+64)
// of L values: out[0] = 0, out[i] = out[i-1] + v[i-1].  Sequential on purpose
// (the rounding of a prefix must not depend on the reduction tree).
__device__ __forceinline__ void seq_prefix(double v0, double v1, int L, int lane, double* out)
{
    double acc = 0.0, r0 = 0.0, r1 = 0.0;
    const int n0 = L < 64 ? L : 64;
    for (int i = 0; i < n0; ++i) {
        acc = acc + bcast(v0, i);
        if (lane == i) r0 = acc;
    }
    for (int i = 64; i < L; ++i) {
        acc = acc + bcast(v1, i - 64);
        if (lane == i - 64) r1 = acc;
    }
    if (lane == 0) out[0] = 0.0;
    if (lane < L) out[lane + 1] = r0;
    if (lane + 64 < L) out[lane + 65] = r1;
}

struct Cell {
    int n;          // GPUs of the cell
    double kappa;   // contention factor of the grid
    double B_pp;    // link between pipeline neighbours
};

struct JobCtx {
    int L, Bg;
    bool moe;       // has all-to-all layers
};

// Per-sample cost of each layer (formula in arena.h), prefix-summed into S.U.
__device__ void build_prefix_u(Lds& S, int lane, const JobCtx& jb, const TypeDev& ty,
                               double kappa, int tp, bool a2a_on)
{
    const double denom = (double)jb.Bg * ty.speed * (double)tp;
    const double ctp = kappa * 8.0 * (double)(tp - 1) / (double)tp;
    double u[2] = {0.0, 0.0};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int l = lane + 64 * s;
        if (l < jb.L) {
            double v = (double)S.t[l] / denom;
            if (tp > 1) v += ctp * (double)S.x[l] / ty.bw_intra;
            if (a2a_on) v += kappa * (double)S.q[l] / ty.bw_inter;
            u[s] = v;
        }
    }
    seq_prefix(u[0], u[1], jb.L, lane, S.U);
    sync();
}

// Pipeline degrees the problem must answer: divisors pp of n/tp with
// pp <= L, at least one admissible microbatch count, and the all-to-all
// condition of the variant.  Writes S.tg ascending, returns how many.
__device__ int build_targets(Lds& S, int lane, const JobCtx& jb, int n, int tp, int variant,
                             const EstimateArgs& A)
{
    const int q = n / tp;
    int nt = 0;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int pp = 1 + lane + 64 * s;
        bool ok = pp <= jb.L && (q % pp) == 0;
        if (ok) ok = (variant == 0) ? (!jb.moe || pp < n) : (pp == n);
        if (ok) {
            const int dp = q / pp;
            bool anym = false;
            for (int i = 0; i < A.n_m; ++i) anym |= (jb.Bg % (dp * A.m_values[i])) == 0;
            ok = anym;
        }
        const unsigned long long mask = __ballot(ok);
        if (ok) S.tg[nt + __popcll(mask & ((1ull << lane) - 1ull))] = pp;
        nt += __popcll(mask);
    }
    sync();
    return nt;
}

// Canonical cuts for degree pp and bottleneck W: c_pp = L and, right to
// left, c_k = max(k, next(c_{k+1})) with next(e) the smallest c such that
// U_e - U_c <= W.  Returns stage bounds in registers: stage s = lane + 64*h
// holds layers [st_h, en_h).
struct Stages {
    int st0, st1, en0, en1;
};

__device__ __forceinline__ void put_stage_start(Stages& r, int lane, int stage, int v)
{
    if (stage < 64) { if (lane == stage) r.st0 = v; }
    else if (lane == stage - 64) r.st1 = v;
}

__device__ __forceinline__ void put_stage_end(Stages& r, int lane, int stage, int v)
{
    if (stage < 64) { if (lane == stage) r.en0 = v; }
    else if (lane == stage - 64) r.en1 = v;
}

__device__ Stages canonical_stages(const Lds& S, int lane, int L, int pp, double W)
{
    int nx0 = 0, nx1 = 0;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int e = 1 + lane + 64 * s;
        if (e <= L) {
            const double Ue = S.U[e];
            int lo = 0, hi = e - 1;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (Ue - S.U[mid] <= W) hi = mid; else lo = mid + 1;
            }
            if (s == 0) nx0 = lo; else nx1 = lo;
        }
    }
    Stages r = {0, 0, 0, 0};
    put_stage_end(r, lane, pp - 1, L);      // stage 0 starts at 0 (already 0)
    int cur = L;
    for (int k = pp - 1; k >= 1; --k) {
        const int e = cur - 1;
        const int nxt = (e < 64) ? __builtin_amdgcn_readlane(nx0, e)
                                 : __builtin_amdgcn_readlane(nx1, e - 64);
        const int c = nxt > k ? nxt : k;
        put_stage_start(r, lane, k, c);
        put_stage_end(r, lane, k - 1, c);
        cur = c;
        if (c == k) {
            // every earlier stage holds exactly one layer
            if (lane < k) { r.st0 = lane; r.en0 = lane + 1; }
            if (lane + 64 < k) { r.st1 = lane + 64; r.en1 = lane + 65; }
            break;
        }
    }
    return r;
}

// Price every admissible microbatch count of plan (dp, tp, pp) given the
// canonical stages; appends to the cell's plan buffer.
__device__ void price_target(Lds& S, int lane, const JobCtx& jb, const TypeDev& ty,
                             const Cell& cell, int tp, int pp, double W, int& np,
                             const EstimateArgs& A, unsigned long long& overflow)
{
    const Stages sg = canonical_stages(S, lane, jb.L, pp, W);

    const int dp = cell.n / (tp * pp);
    const int grp = dp * tp;
    const double B_dp = (grp <= ty.gpn && ty.gpn % grp == 0) ? ty.bw_intra : ty.bw_inter;

    double Sk[2], Pk[2], Ak[2], xk[2];
    bool act[2];
    double pmax = 0.0;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int stage = lane + 64 * s;
        act[s] = stage < pp;
        Sk[s] = Pk[s] = Ak[s] = xk[s] = 0.0;
        if (act[s]) {
            const int lo = s == 0 ? sg.st0 : sg.st1;
            const int hi = s == 0 ? sg.en0 : sg.en1;
            Sk[s] = S.U[hi] - S.U[lo];
            Pk[s] = S.Pp[hi] - S.Pp[lo];
            Ak[s] = S.Ap[hi] - S.Ap[lo];
            xk[s] = (stage < pp - 1) ? (double)S.x[hi - 1] : 0.0;
            pmax = fmax(pmax, Pk[s]);
        }
    }
    pmax = wave_max(pmax);
    const double ar = (dp > 1)
        ? cell.kappa * 2.0 * (double)(dp - 1) / (double)dp * (pmax / (double)tp) / B_dp
        : 0.0;

    for (int mi = 0; mi < A.n_m; ++mi) {
        const int m = A.m_values[mi];
        if (jb.Bg % (dp * m) != 0) continue;
        const double b = (double)jb.Bg / (double)(dp * m);
        double fill = 0.0, mem = 0.0;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            if (!act[s]) continue;
            const int stage = lane + 64 * s;
            const double Wk = b * Sk[s];
            const double p2p = (stage < pp - 1) ? cell.kappa * 2.0 * b * xk[s] / cell.B_pp : 0.0;
            fill += Wk + p2p;
            const int inflight = m < pp - stage ? m : pp - stage;
            const double Mk = 4.0 * Pk[s] / (double)tp + (double)inflight * b * Ak[s] / (double)tp;
            mem = fmax(mem, Mk);
        }
        fill = wave_sum(fill);
        mem = wave_max(mem);
        const double wmax = b * W;
        const double T = fill + (double)(m - 1) * wmax + ar;
        if (np < kMaxPlans) {
            if (lane == 0) {
                S.planT[np] = (mem <= ty.mem) ? T : kInf;
                S.planW[np] = W;
                S.planKey[np] = ((unsigned)pp << 16) | ((unsigned)tp << 8) | (unsigned)m;
            }
            ++np;
        } else {
            overflow = 1;
        }
    }
}

// Solve one partition problem: the recursion D_k(i) = min over j of
// max(D_{k-1}(j), U_i - U_j), row by row, lanes over i.  The crossing j where
// D_{k-1}(j) >= U_i - U_j first holds never moves left as i or k grows, so
// each lane keeps its crossing from row to row and only walks it forward.
// Row k is evaluated for i in [k, L - tau(k) + k] only, tau(k) being the
// smallest requested degree >= k (larger i cannot reach a requested cell).
__device__ void solve_problem(Lds& S, int lane, const JobCtx& jb, const TypeDev& ty,
                              const Cell& cell, int tp, int nt, int& np,
                              const EstimateArgs& A, unsigned long long& dp_entries,
                              unsigned long long& overflow)
{
    const int L = jb.L;
    double* Dp = S.D[0];
    double* Dc = S.D[1];
    int ti = 0;
    int tau = S.tg[0];
    const int P = S.tg[nt - 1];
    int jp[2] = {0, 0};

    // row 1
    {
        const int hi = L - tau + 1;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int i = 1 + lane + 64 * s;
            if (i <= hi) Dc[i] = S.U[i];
        }
        dp_entries += (unsigned long long)hi;
        sync();
        double* tmp = Dp; Dp = Dc; Dc = tmp;
        if (tau == 1) {
            price_target(S, lane, jb, ty, cell, tp, 1, Dp[L], np, A, overflow);
            ++ti;
            tau = ti < nt ? S.tg[ti] : 0;
        }
    }
    for (int k = 2; k <= P; ++k) {
        const int hi = L - tau + k;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int i = 1 + lane + 64 * s;
            if (i >= k && i <= hi) {
                const double Ui = S.U[i];
                int j = jp[s] > k - 1 ? jp[s] : k - 1;
                while (j < i) {
                    if (Dp[j] >= Ui - S.U[j]) break;
                    ++j;
                }
                jp[s] = j;
                double v = (j < i) ? Dp[j] : kInf;
                if (j - 1 >= k - 1) v = fmin(v, Ui - S.U[j - 1]);
                Dc[i] = v;
            }
        }
        dp_entries += (unsigned long long)(hi - k + 1);
        sync();
        double* tmp = Dp; Dp = Dc; Dc = tmp;
        if (k == tau) {
            price_target(S, lane, jb, ty, cell, tp, k, Dp[L], np, A, overflow);
            ++ti;
            tau = ti < nt ? S.tg[ti] : 0;
        }
    }
    sync();
}

__global__ __launch_bounds__(64) void estimate_kernel(EstimateArgs A)
{
    __shared__ Lds S;
    const int lane = threadIdx.x;
    const int item = blockIdx.x;
    const int j = item / A.n_types;
    const int g = item - j * A.n_types;

    const int off = A.layer_offset[j];
    JobCtx jb;
    jb.L = A.layer_offset[j + 1] - off;
    jb.Bg = A.batch[j];
    const TypeDev ty = A.types[g];

    // stage the job
    bool has_q = false;
    double pv[2] = {0.0, 0.0}, av[2] = {0.0, 0.0};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int l = lane + 64 * s;
        if (l < jb.L) {
            S.t[l] = A.t[off + l];
            S.x[l] = A.x[off + l];
            const float qv = A.q[off + l];
            S.q[l] = qv;
            has_q |= qv > 0.0f;
            pv[s] = (double)A.p[off + l];
            av[s] = (double)A.a[off + l];
        }
    }
    jb.moe = __ballot(has_q) != 0ull;
    seq_prefix(pv[0], pv[1], jb.L, lane, S.Pp);
    seq_prefix(av[0], av[1], jb.L, lane, S.Ap);
    sync();

    unsigned long long n_plans = 0, n_problems = 0, dp_entries = 0, n_infeasible = 0, overflow = 0;

    for (int ci = 0; ci < A.n_counts; ++ci) {
        Cell cell;
        cell.n = A.counts[ci];
        cell.kappa = (double)A.kappa[g * A.n_counts + ci];
        cell.B_pp = (cell.n <= ty.gpn) ? ty.bw_intra : ty.bw_inter;
        int np = 0;

        const int tpmax = cell.n < ty.gpn ? cell.n : ty.gpn;
        for (int tp = 1; tp <= tpmax; ++tp) {
            if (cell.n % tp != 0 || ty.gpn % tp != 0) continue;
            for (int variant = 0; variant < 2; ++variant) {
                if (variant == 1 && !(jb.moe && tp == 1)) break;
                const int nt = build_targets(S, lane, jb, cell.n, tp, variant, A);
                if (nt == 0) continue;
                build_prefix_u(S, lane, jb, ty, cell.kappa, tp, variant == 0);
                solve_problem(S, lane, jb, ty, cell, tp, nt, np, A, dp_entries, overflow);
                ++n_problems;
            }
        }
        sync();

        // best plan of the cell: smallest key among plans within the tie window
        double tl = kInf;
        for (int e = lane; e < np; e += 64) tl = fmin(tl, S.planT[e]);
        const double tmin = wave_min(tl);
        const long long cidx = ((long long)j * A.n_types + g) * A.n_counts + ci;
        n_plans += (unsigned long long)np;
        if (!(tmin < kInf)) {
            ++n_infeasible;
            if (lane == 0) {
                A.t_iter[cidx] = __builtin_huge_valf();
                A.thr[cidx] = 0.0f;
                A.plan[cidx] = 0u;
            }
            if (A.cuts) {
                uint8_t* row = A.cuts + cidx * A.cuts_stride;
                for (int e = lane; e < A.cuts_stride; e += 64) row[e] = 0xFF;
            }
            sync();
            continue;
        }
        const double lim = tmin * (1.0 + A.tie_eps);
        unsigned kl = 0xFFFFFFFFu;
        for (int e = lane; e < np; e += 64)
            if (S.planT[e] <= lim) kl = S.planKey[e] < kl ? S.planKey[e] : kl;
        const unsigned kbest = wave_min_u(kl);
        int il = -1;
        for (int e = lane; e < np; e += 64)
            if (S.planKey[e] == kbest) il = e;
        const int ib = wave_max_i(il);
        const double Tb = S.planT[ib];
        const double Wb = S.planW[ib];
        const int pp = (int)(kbest >> 16);
        const int tp = (int)((kbest >> 8) & 0xFFu);
        const int m = (int)(kbest & 0xFFu);
        const int dp = cell.n / (tp * pp);
        if (lane == 0) {
            A.t_iter[cidx] = (float)Tb;
            A.thr[cidx] = (float)((double)jb.Bg / Tb);
            A.plan[cidx] = (unsigned)dp | ((unsigned)tp << 11) | ((unsigned)pp << 16) |
                           ((unsigned)m << 24) | (1u << 31);
        }
        if (A.cuts) {
            const bool a2a_on = !jb.moe || dp * tp > 1;
            build_prefix_u(S, lane, jb, ty, cell.kappa, tp, a2a_on);
            const Stages sg = canonical_stages(S, lane, jb.L, pp, Wb);
            uint8_t* row = A.cuts + cidx * A.cuts_stride;
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const int idx = lane + 64 * s;
                const int en = s == 0 ? sg.en0 : sg.en1;
                if (idx < A.cuts_stride) row[idx] = (idx < pp - 1) ? (uint8_t)en : (uint8_t)0xFF;
            }
            for (int e = 128 + lane; e < A.cuts_stride; e += 64) row[e] = 0xFF;
        }
        sync();
    }

    if (lane == 0) {
        atomicAdd(&A.counters[kCells], (unsigned long long)A.n_counts);
        atomicAdd(&A.counters[kPlans], n_plans);
        atomicAdd(&A.counters[kProblems], n_problems);
        atomicAdd(&A.counters[kDpEntries], dp_entries);
        atomicAdd(&A.counters[kInfeasible], n_infeasible);
        if (overflow) atomicAdd(&A.counters[kOverflow], 1ull);
    }
}

__global__ void zero_kernel(unsigned long long* p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0ull;
}

// One wave per job: every per-layer value must be finite and >= 0.
__global__ __launch_bounds__(64) void validate_kernel(ValidateArgs V)
{
    const int j = blockIdx.x;
    const int lane = threadIdx.x;
    const int lo = V.layer_offset[j], hi = V.layer_offset[j + 1];
    unsigned bad = 0;
    for (int l = lo + lane; l < hi; l += 64) {
#pragma unroll
        for (int k = 0; k < 5; ++k) {
            const float v = V.arrays[k][l];
            if (!(v >= 0.0f) || !(v <= 3.402823466e38f)) ++bad;
        }
    }
    if (bad) atomicAdd(V.bad, (unsigned long long)bad);
}

}  // namespace

hipError_t launch_estimate(const EstimateArgs& args, hipStream_t stream)
{
    const long long blocks = (long long)args.n_jobs * args.n_types;
    if (blocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(estimate_kernel, dim3((unsigned)blocks), dim3(64), 0, stream, args);
    return hipGetLastError();
}

hipError_t launch_zero_counters(unsigned long long* counters, int n, hipStream_t stream)
{
    hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(64), 0, stream, counters, n);
    return hipGetLastError();
}

hipError_t launch_validate(const ValidateArgs& args, hipStream_t stream)
{
    if (args.n_jobs <= 0) return hipSuccess;
    hipLaunchKernelGGL(validate_kernel, dim3((unsigned)args.n_jobs), dim3(64), 0, stream, args);
    return hipGetLastError();
}

}  // namespace arena
