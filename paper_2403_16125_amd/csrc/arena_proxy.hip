// HIP kernel of the proxy-plan planner (gfx950).
//
// For every (job, GPU type, GPU count) cell, the load-aware planner of
// Sec. 3.3 without execution:
//   * the job's layers form O = min(L, n_ops) clustered operators; each
//     operator's load is its roofline time (Eq. 2: FLOPs over the attainable
//     rate at its arithmetic intensity) and its GPU share is proportional to
//     the load;
//   * every pipeline degree s is a grid (Sec. 3.2); in it every contiguous
//     grouping of the operators into s stages is normalised to power-of-two
//     stage GPU counts summing to n with the least computation bias (Eq. 3);
//   * per microbatch count B, among groupings whose stages fit memory, the
//     proxy plan has the least bias, then the least communication load
//     (Eq. 4) with each stage's intra-stage (dp, tp) chosen for the least
//     communication; it is priced by the 1F1B model with per-stage GPU
//     counts (Sec. 3.4);
//   * the cell keeps the fastest grid (ties within the tie window: fewer
//     stages, then fewer microbatches).
//
// One workgroup of 4 waves per cell.  Within a grid the groupings are
// ranked in lexicographic order of their cut vectors and spread over the
// threads: each unranks its grouping, sums the stage shares, ranks the
// stages, scans the power-of-two multisets of (n, s) -- staged in LDS,
// lexicographically descending, so the first least cost wins ties -- and
// tests every B for memory with the largest admissible tensor degree
// (memory falls with tp and admissibility only gets easier, so that tp fits
// iff some tp does).  Bias and feasibility are kept per grouping in LDS;
// each B is then a block-wide arg-min.  Arithmetic is fp64 in the operation
// order of a plain evaluation (left-to-right stage sums, the bias summed
// over stages in stage order), so every decision is reproducible.
#include <math.h>

#include "arena_internal.h"

namespace arena {
namespace {

constexpr int kPxThreads = 1024;
constexpr int kPxWaves = kPxThreads / 64;
constexpr int kMaxParts = 6435;           // C(15, 7): groupings of 16 operators
constexpr double kInfP = __builtin_huge_val();

struct ProxyLds {
    unsigned long long ms[kProxyMaxMultisets];   // multisets of the current (n, s)
    double b2[kMaxParts];                        // least squared bias of each grouping
    uint16_t fmask[kMaxParts];                   // bit k: every stage fits at m_values[k]
    uint16_t bestk[kMaxParts];                   // its least-bias multiset
    // operator sums (left to right over their layers)
    double od[kProxyMaxOps], oT[kProxyMaxOps], oX[kProxyMaxOps], oE[kProxyMaxOps];
    double oP[kProxyMaxOps], oA[kProxyMaxOps], oxl[kProxyMaxOps], oload[kProxyMaxOps];
    int32_t binom[16][16];
    int32_t mval[kMaxM];
    double bt[11][kMaxM];                        // replica samples at dp = 2^e, m_values[k]; -1: not a divisor
    double gT[kProxyMaxOps + 1][kMaxM];          // T of each grid's proxy (inf: none fits)
    int32_t gR[kProxyMaxOps + 1][kMaxM];         // its grouping rank
    unsigned long long gD[kProxyMaxOps + 1][kMaxM];   // its stage GPU exponents
    unsigned long long gP[kProxyMaxOps + 1][kMaxM];   // its stage tensor-degree exponents
    // left-to-right sums of the operator quantities over every operator range
    // [lo, hi): ss[quantity][lo * 17 + hi]
    double ss[6][17 * 17];
    double rkey[kPxWaves];
    int32_t ridx[kPxWaves];
    double wkey[kPxWaves][kMaxM];                // per-wave minima of every B
    int32_t widx[kPxWaves][kMaxM];
    double minb2[kMaxM];                         // least bias that fits, per B
    int32_t win[kMaxM];                          // its grouping (after the ties)
    uint32_t tiemask;                            // B with another grouping of equal bias
    int32_t rflag;
    int32_t no_load;                             // every operator has zero load: no proxy plan
};

// The cell's constants.
struct Cell {
    int L, Bg, O, n, gpn;
    double speed, mem, bwi, bwe, kap;
};

// (key, idx) of another lane picked by one DPP control; lanes of the rows
// the row mask leaves out read the identity (+inf, INT_MAX).
template <int CTRL, int ROWS>
__device__ __forceinline__ void dpp_pair(double k, int i, double& ok, int& oi)
{
    const unsigned long long b = (unsigned long long)__double_as_longlong(k);
    const unsigned long long e = (unsigned long long)__double_as_longlong(kInfP);
    const int lo = __builtin_amdgcn_update_dpp((int)(unsigned)e, (int)(unsigned)b, CTRL, ROWS, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(unsigned)(e >> 32), (int)(unsigned)(b >> 32), CTRL, ROWS,
                                               0xf, false);
    ok = __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) |
                                          (unsigned long long)(unsigned)lo));
    oi = __builtin_amdgcn_update_dpp(0x7fffffff, i, CTRL, ROWS, 0xf, false);
}

__device__ __forceinline__ void take_less(double& k, int& i, double ok, int oi)
{
    const bool t = (ok < k) | ((ok == k) & (oi < i));
    k = t ? ok : k;
    i = t ? oi : i;
}

// Least (key, idx) of the wave (smaller key, then smaller idx), in every
// lane: quad swaps and row rotations give each row its least pair, row
// broadcasts carry it to the last row, lane 63 hands the result out.  DPP
// moves need no lane addresses (a shuffle's would be held in registers).
__device__ __forceinline__ void wave_argmin(double& k, int& i)
{
    double ok;
    int oi;
    dpp_pair<0xB1, 0xf>(k, i, ok, oi);    // quad_perm [1,0,3,2]
    take_less(k, i, ok, oi);
    dpp_pair<0x4E, 0xf>(k, i, ok, oi);    // quad_perm [2,3,0,1]
    take_less(k, i, ok, oi);
    dpp_pair<0x124, 0xf>(k, i, ok, oi);   // row_ror:4
    take_less(k, i, ok, oi);
    dpp_pair<0x128, 0xf>(k, i, ok, oi);   // row_ror:8
    take_less(k, i, ok, oi);
    dpp_pair<0x142, 0xa>(k, i, ok, oi);   // row_bcast:15 into rows 1 and 3
    take_less(k, i, ok, oi);
    dpp_pair<0x143, 0xc>(k, i, ok, oi);   // row_bcast:31 into rows 2 and 3
    take_less(k, i, ok, oi);
    const unsigned long long b = (unsigned long long)__double_as_longlong(k);
    const int lo = __builtin_amdgcn_readlane((int)(unsigned)b, 63);
    const int hi = __builtin_amdgcn_readlane((int)(unsigned)(b >> 32), 63);
    k = __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) |
                                         (unsigned long long)(unsigned)lo));
    i = __builtin_amdgcn_readlane(i, 63);
}

// Block-wide arg-min of (key, idx) (smaller key, then smaller idx).
__device__ __forceinline__ void block_argmin(double& key, int& idx, ProxyLds& S)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    wave_argmin(key, idx);
    if (lane == 0) {
        S.rkey[w] = key;
        S.ridx[w] = idx;
    }
    __syncthreads();
    key = S.rkey[0];
    idx = S.ridx[0];
#pragma unroll
    for (int q = 1; q < kPxWaves; ++q) {
        const double ok = S.rkey[q];
        const int oi = S.ridx[q];
        if (ok < key || (ok == key && oi < idx)) {
            key = ok;
            idx = oi;
        }
    }
    __syncthreads();
}

// Stage-start mask (bit i: a stage starts at operator i, i >= 1) of the
// grouping of rank r among those of O operators into s stages, cut vectors
// in lexicographic order.
__device__ __forceinline__ unsigned unrank(int r, int O, int s, const ProxyLds& S)
{
    unsigned mask = 0u;
    const int N = O - 1, t = s - 1;
    int c = 1;
    for (int q = 0; q < t; ++q) {
        for (;;) {
            const int cnt = S.binom[N - c][t - 1 - q];
            if (r < cnt) break;
            r -= cnt;
            ++c;
        }
        mask |= 1u << c;
        ++c;
    }
    return mask;
}

// The grouping after `mask` in lexicographic order of cut vectors (t cuts
// among operators 1..O-1): the last cut moves up if it can; otherwise the
// cuts packed against the end follow the highest cut that can still move.
__device__ __forceinline__ unsigned next_grouping(unsigned mask, int O, int t)
{
    const int top = O - 1;
    int r = 0;
    while (r < t && ((mask >> (top - r)) & 1u)) ++r;
    if (r == 0) {
        const int c = 31 - __clz(mask);
        return mask ^ (1u << c) ^ (1u << (c + 1));
    }
    const unsigned rest = mask & ~(((1u << r) - 1u) << (top - r + 1));
    const int c = 31 - __clz(rest);
    return (rest ^ (1u << c)) | (1u << (c + 1)) | (((1u << r) - 1u) << (c + 2));
}

// End (exclusive) of the stage starting at `lo`: the next stage start, or O.
__device__ __forceinline__ int stage_end(unsigned mask, int lo, int O)
{
    const unsigned rest = mask & ~((2u << lo) - 1u);
    return rest ? __ffs(rest) - 1 : O;
}

// Operator quantities kept as range sums.
enum { kQd = 0, kQT, kQX, kQE, kQP, kQA };

__device__ __forceinline__ double ssum(const ProxyLds& S, int qn, int lo, int hi)
{
    return S.ss[qn][lo * 17 + hi];
}

// Stage shares D_j (stage order) and each stage's sorted position q_j
// (largest share first, ties to the lower stage); static indices so both
// stay in registers.
__device__ __forceinline__ void shares(unsigned mask, int s, int O, const ProxyLds& S, double (&D)[16],
                                       int (&q)[16])
{
    int lo = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        if (j < s) {
            const int hi = stage_end(mask, lo, O);
            D[j] = ssum(S, kQd, lo, hi);
            lo = hi;
        } else {
            D[j] = 0.0;
        }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        int r = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if (i < s && i != j && (D[i] > D[j] || (D[i] == D[j] && i < j))) ++r;
        q[j] = r;
    }
}

// Squared bias of multiset m (exponents at bits 4p, largest first) with
// stage j taking position q_j, summed over the stages in stage order (S
// stages, a compile-time count so the sum has no branches).
template <int S>
__device__ __forceinline__ double bias(unsigned long long m, const double (&D)[16], const int (&q)[16])
{
    const unsigned lo = (unsigned)m, hi = (unsigned)(m >> 32);
    double cost = 0.0;
#pragma unroll
    for (int j = 0; j < S; ++j) {
        // the exponent of position q_j, then 2^e from its exponent field (e <= 10)
        const unsigned e = __builtin_amdgcn_ubfe(q[j] < 8 ? lo : hi, (unsigned)(4 * q[j]) & 31u, 4u);
        const double diff = __hiloint2double((int)((e << 20) + 0x3ff00000u), 0) - D[j];   // 2^e - share
        cost += diff * diff;
    }
    return cost;
}

// The least bias over multisets k = first, first + step, ... below K (the
// table is lexicographically descending, so among equal costs the smallest k
// wins) and that k (-1 if none).
template <int S>
__device__ __forceinline__ double normalise_s(const double (&D)[16], const int (&q)[16], int K, int first,
                                              int step, const ProxyLds& Ls, int& bk)
{
    double best = kInfP;
    bk = -1;
    // two multisets per iteration (independent sums), compared in order
    int k = first;
    for (; k + step < K; k += 2 * step) {
        const unsigned long long m0 = Ls.ms[k], m1 = Ls.ms[k + step];
        const double c0 = bias<S>(m0, D, q);
        const double c1 = bias<S>(m1, D, q);
        if (c0 < best) {
            best = c0;
            bk = k;
        }
        if (c1 < best) {
            best = c1;
            bk = k + step;
        }
    }
    if (k < K) {
        const double c0 = bias<S>(Ls.ms[k], D, q);
        if (c0 < best) {
            best = c0;
            bk = k;
        }
    }
    return best;
}

// shares() for a compile-time stage count.
template <int S>
__device__ __forceinline__ void shares_s(unsigned mask, int O, const ProxyLds& Ls, double (&D)[16], int (&q)[16])
{
    int lo = 0;
#pragma unroll
    for (int j = 0; j < S; ++j) {
        const int hi = stage_end(mask, lo, O);
        D[j] = ssum(Ls, kQd, lo, hi);
        lo = hi;
    }
#pragma unroll
    for (int j = 0; j < S; ++j) {
        int r = 0;
#pragma unroll
        for (int i = 0; i < S; ++i)
            if (i != j && (D[i] > D[j] || (D[i] == D[j] && i < j))) ++r;
        q[j] = r;
    }
}

// One grouping's shares, ranks and least bias (over its lane's multisets).
template <int S>
__device__ __forceinline__ double group_bias(unsigned mask, int O, int K, int first, int step, const ProxyLds& Ls,
                                             double (&D)[16], int (&q)[16], int& bk)
{
    shares_s<S>(mask, O, Ls, D, q);
    return normalise_s<S>(D, q, K, first, step, Ls, bk);
}

__device__ __forceinline__ double group_bias(int s, unsigned mask, int O, int K, int first, int step,
                                             const ProxyLds& Ls, double (&D)[16], int (&q)[16], int& bk)
{
    switch (s) {
#define ARENA_PX_CASE(n) case n: return group_bias<n>(mask, O, K, first, step, Ls, D, q, bk);
        ARENA_PX_CASE(1) ARENA_PX_CASE(2) ARENA_PX_CASE(3) ARENA_PX_CASE(4)
        ARENA_PX_CASE(5) ARENA_PX_CASE(6) ARENA_PX_CASE(7) ARENA_PX_CASE(8)
        ARENA_PX_CASE(9) ARENA_PX_CASE(10) ARENA_PX_CASE(11) ARENA_PX_CASE(12)
        ARENA_PX_CASE(13) ARENA_PX_CASE(14) ARENA_PX_CASE(15) ARENA_PX_CASE(16)
#undef ARENA_PX_CASE
        default: bk = -1; return kInfP;
    }
}

// The stage exponents (4 bits per stage, stage order) multiset m assigns.
__device__ __forceinline__ unsigned long long stage_exps(unsigned long long m, const int (&q)[16], int s)
{
    unsigned long long dexp = 0ull;
#pragma unroll
    for (int j = 0; j < 16; ++j)
        if (j < s) dexp |= ((m >> (4 * q[j])) & 15ull) << (4 * j);
    return dexp;
}

// Per-replica samples of a stage with D GPUs at tensor degree tp and B
// microbatches, or -1 when dp B does not divide the batch.
__device__ __forceinline__ double replica_batch(int Bg, int D, int tp, int B)
{
    const int dp = D / tp;
    if (Bg % (dp * B)) return -1.0;
    return (double)Bg / (double)(dp * B);
}

__device__ __forceinline__ double stage_mem(double P, double A, int tp, double b, int inflight)
{
    return 4.0 * P / (double)tp + (double)inflight * b * A / (double)tp;
}

// Intra-stage communication per microbatch (C) and gradient all-reduce per
// iteration (AR) of a stage with operator range [lo, hi), D GPUs, degree tp.
__device__ __forceinline__ void stage_comm(const Cell c, const ProxyLds& S, int lo, int hi, int D, int tp,
                                           double b, double& C, double& AR)
{
    const double X = ssum(S, kQX, lo, hi), E = ssum(S, kQE, lo, hi), P = ssum(S, kQP, lo, hi);
    double per_sample = 0.0;
    if (tp > 1) per_sample += c.kap * 8.0 * (double)(tp - 1) / (double)tp * X / c.bwi;
    if (D > 1) per_sample += c.kap * E / c.bwe;
    C = b * per_sample;
    const int dp = D / tp;
    const double B_dp = (D <= c.gpn && c.gpn % D == 0) ? c.bwi : c.bwe;
    AR = 0.0;
    if (dp > 1) AR = c.kap * 2.0 * (double)(dp - 1) / (double)dp * (P / (double)tp) / B_dp;
}

// Every stage's tp (least communication B C + AR within memory, ties to the
// smaller tp) and the communication load (Eq. 4); false if a stage has none.
__device__ __forceinline__ bool plan_lcomm(const Cell c, const ProxyLds& S, unsigned mask, int s, int B,
                           unsigned long long dexp, unsigned long long& texp, double& lcomm)
{
    double cmax = 0.0, csum = 0.0, arsum = 0.0;
    texp = 0ull;
    int lo = 0;
    for (int j = 0; j < s; ++j) {
        const int hi = stage_end(mask, lo, c.O);
        const int D = 1 << (int)((dexp >> (4 * j)) & 15ull);
        const int inflight = B < s - j ? B : s - j;
        const double P = ssum(S, kQP, lo, hi), A = ssum(S, kQA, lo, hi);
        int best = 0;
        double best_cost = 0.0, bC = 0.0, bAR = 0.0;
        for (int tp = 1; tp <= D; tp *= 2) {
            if (D % tp || c.gpn % tp) continue;
            const double b = replica_batch(c.Bg, D, tp, B);
            if (b < 0.0) continue;
            if (stage_mem(P, A, tp, b, inflight) > c.mem) continue;
            double C, AR;
            stage_comm(c, S, lo, hi, D, tp, b, C, AR);
            const double cost = (double)B * C + AR;
            if (best == 0 || cost < best_cost) {
                best = tp;
                best_cost = cost;
                bC = C;
                bAR = AR;
            }
        }
        if (best == 0) return false;
        texp |= (unsigned long long)(__ffs(best) - 1) << (4 * j);
        if (bC > cmax) cmax = bC;
        csum += bC;
        arsum += bAR;
        lo = hi;
    }
    lcomm = (double)(B - 1) * cmax + csum + arsum;
    return true;
}

// The 1F1B iteration time with per-stage (dp_j, tp_j).
__device__ __forceinline__ double price(const Cell c, const ProxyLds& S, unsigned mask, int s, int B, unsigned long long dexp,
                        unsigned long long texp)
{
    const double B_pp = (c.n <= c.gpn) ? c.bwi : c.bwe;
    double fill = 0.0, wmax = 0.0, armax = 0.0;
    int lo = 0;
    for (int j = 0; j < s; ++j) {
        const int hi = stage_end(mask, lo, c.O);
        const int D = 1 << (int)((dexp >> (4 * j)) & 15ull);
        const int tp = 1 << (int)((texp >> (4 * j)) & 15ull);
        const int dp = D / tp;
        const double b = replica_batch(c.Bg, D, tp, B);
        if (b < 0.0) return kInfP;
        const int inflight = B < s - j ? B : s - j;
        const double T = ssum(S, kQT, lo, hi), X = ssum(S, kQX, lo, hi), E = ssum(S, kQE, lo, hi);
        const double P = ssum(S, kQP, lo, hi), A = ssum(S, kQA, lo, hi);
        if (stage_mem(P, A, tp, b, inflight) > c.mem) return kInfP;
        double per_sample = T / ((double)c.Bg * c.speed * (double)tp);
        if (tp > 1) per_sample += c.kap * 8.0 * (double)(tp - 1) / (double)tp * X / c.bwi;
        if (D > 1) per_sample += c.kap * E / c.bwe;
        const double W = b * per_sample;
        double p2p = 0.0;
        if (j < s - 1) {
            const int Dn = 1 << (int)((dexp >> (4 * (j + 1))) & 15ull);
            const int tpn = 1 << (int)((texp >> (4 * (j + 1))) & 15ull);
            const int dpn = Dn / tpn;
            const int dmin = dp < dpn ? dp : dpn;
            p2p = c.kap * 2.0 * ((double)c.Bg / (double)(dmin * B)) * S.oxl[hi - 1] / B_pp;
        }
        const double B_dp = (D <= c.gpn && c.gpn % D == 0) ? c.bwi : c.bwe;
        double AR = 0.0;
        if (dp > 1) AR = c.kap * 2.0 * (double)(dp - 1) / (double)dp * (P / (double)tp) / B_dp;
        fill += W + p2p;
        if (W > wmax) wmax = W;
        if (AR > armax) armax = AR;
        lo = hi;
    }
    return fill + (double)(B - 1) * wmax + armax;
}

__device__ __forceinline__ void proxy_cell(const ProxyArgs& A, ProxyLds& S, int cell)
{
    // the thread index passes through an empty asm statement once per cell, so
    // nothing derived from it is hoisted out of the cell loop and held in
    // registers across every cell (it would be spilled)
    int tid;
    __asm__ volatile("" : "=v"(tid) : "0"((int)threadIdx.x));
    const int ci = cell % A.n_counts;
    const int g = (cell / A.n_counts) % A.n_types;
    const int jb = cell / (A.n_counts * A.n_types);

    Cell c;
    const int off0 = A.layer_offset[jb];
    c.L = A.layer_offset[jb + 1] - off0;
    c.Bg = A.batch[jb];
    c.O = c.L < A.n_ops ? c.L : A.n_ops;
    c.n = A.counts[ci];
    const TypeDev ty = A.types[g];
    c.speed = ty.speed;
    c.mem = ty.mem;
    c.bwi = ty.bw_intra;
    c.bwe = ty.bw_inter;
    c.gpn = ty.gpn;
    c.kap = (double)A.kappa[g * A.n_counts + ci];
    const double hbm = A.hbm[g];

    // operator sums, loads and shares; binomials; microbatch counts
    if (tid < c.O) {
        const int lo = (int)(((long long)tid * c.L) / c.O), hi = (int)(((long long)(tid + 1) * c.L) / c.O);
        double T = 0.0, X = 0.0, E = 0.0, P = 0.0, Ac = 0.0, M = 0.0;
        for (int l = off0 + lo; l < off0 + hi; ++l) {
            T += (double)A.t[l];
            X += (double)A.x[l];
            E += (double)A.q[l];
            P += (double)A.p[l];
            Ac += (double)A.a[l];
            M += (double)A.p[l] + (double)c.Bg * (double)A.a[l];
        }
        S.oT[tid] = T;
        S.oX[tid] = X;
        S.oE[tid] = E;
        S.oP[tid] = P;
        S.oA[tid] = Ac;
        S.oxl[tid] = (double)A.x[off0 + hi - 1];
        const double flops = A.f_ref * T;
        const double compute = flops / (c.speed * A.f_ref);
        const double memory = M / hbm;
        S.oload[tid] = compute > memory ? compute : memory;
    }
    if (tid < 256) {
        const int a = tid >> 4, b = tid & 15;
        int v = 0;
        if (b <= a) {          // C(a, b) by the multiplicative formula (exact in 32 bits for a <= 15)
            v = 1;
            for (int k = 1; k <= b; ++k) v = v * (a - b + k) / k;
        }
        S.binom[a][b] = v;
    }
    if (tid < A.n_m) S.mval[tid] = A.m_values[tid];
    if (tid < 11 * A.n_m) {
        const int e = tid / A.n_m, k = tid - e * A.n_m;
        S.bt[e][k] = replica_batch(c.Bg, 1 << e, 1, A.m_values[k]);
    }
    for (int z = tid; z < (kProxyMaxOps + 1) * kMaxM; z += kPxThreads) {
        (&S.gT[0][0])[z] = kInfP;
        (&S.gR[0][0])[z] = -1;
    }
    __syncthreads();
    if (tid == 0) {
        double lsum = 0.0;
        for (int i = 0; i < c.O; ++i) lsum += S.oload[i];
        for (int i = 0; i < c.O; ++i) S.od[i] = (S.oload[i] / lsum) * (double)c.n;
        S.no_load = lsum > 0.0 ? 0 : 1;
    }
    __syncthreads();
    for (int task = tid; task < 6 * 17 * 17; task += kPxThreads) {
        const int qn = task / 289, rr = task - qn * 289, lo = rr / 17, hi = rr - lo * 17;
        const double* v = qn == kQd ? S.od : qn == kQT ? S.oT : qn == kQX ? S.oX : qn == kQE ? S.oE
                         : qn == kQP ? S.oP : S.oA;
        double acc = 0.0;
        if (lo < hi && hi <= c.O)
            for (int i = lo; i < hi; ++i) acc += v[i];
        S.ss[qn][rr] = acc;
    }
    __syncthreads();

    const int smax = S.no_load ? 0 : (c.O < c.n ? c.O : c.n);
    const int gpe = __ffs(c.gpn) - 1;             // log2 of the largest power of two dividing the node size
    for (int s = 1; s <= smax; ++s) {
        const int mo = A.mset_off[ci * 17 + s];
        const int K = A.mset_off[ci * 17 + s + 1] - mo;
        if (K <= 0) continue;                      // no s powers of two sum to n
        for (int k = tid; k < K; k += kPxThreads) S.ms[k] = A.msets[mo + k];
        __syncthreads();
        const int nparts = S.binom[c.O - 1][s - 1];
        // a group of tpg lanes (a power of two within one wave) per grouping,
        // each scanning every tpg-th multiset, so few groupings with many
        // multisets still fill the block
        int tpg = 1;
        while (tpg < 64 && tpg * 2 * nparts <= kPxThreads) tpg *= 2;
        const int sub = tid & (tpg - 1);
        const int slots = kPxThreads / tpg;
        // each slot takes a run of consecutive ranks: unrank the first, step to the next
        const int chunk = (nparts + slots - 1) / slots;
        const int r0 = (tid / tpg) * chunk;
        unsigned mask = 0u;
        for (int it = 0; it < chunk; ++it) {
            const int r = r0 + it;
            const bool live = r < nparts;
            double D[16];
            int q[16];
            double best = kInfP;
            int bk = 0x7fffffff;
            if (live) {
                mask = it == 0 ? unrank(r, c.O, s, S) : next_grouping(mask, c.O, s - 1);
                int kk;
                best = group_bias(s, mask, c.O, K, sub, tpg, S, D, q, kk);
                if (kk >= 0) bk = kk;
            }
            for (int off = 1; off < tpg; off <<= 1) {
                const double ob = __shfl_xor(best, off);
                const int ok = __shfl_xor(bk, off);
                if (ob < best || (ob == best && ok < bk)) {
                    best = ob;
                    bk = ok;
                }
            }
            if (live && sub == 0) {
                const unsigned long long dexp = stage_exps(S.ms[bk], q, s);
                // memory test per B at the largest admissible tensor degree
                // (replica samples from the per-cell table; dividing by the
                // power-of-two tp is scaling by its exact reciprocal, so the
                // memory is bitwise the plain formula's)
                unsigned fm = (1u << A.n_m) - 1u;
                int lo = 0;
                for (int j = 0; j < s && fm; ++j) {
                    const int hi = stage_end(mask, lo, c.O);
                    const int ej = (int)((dexp >> (4 * j)) & 15ull);
                    const int te = ej < gpe ? ej : gpe;                  // log2 of the largest tp
                    const double itp = __hiloint2double((1023 - te) << 20, 0);
                    const double P = ssum(S, kQP, lo, hi), Aj = ssum(S, kQA, lo, hi);
                    const double pmem = 4.0 * P * itp;
                    const double* bt = S.bt[ej - te];
                    for (int k = 0; k < A.n_m; ++k) {
                        if (!((fm >> k) & 1u)) continue;
                        const int B = S.mval[k];
                        const double b = bt[k];
                        const int inflight = B < s - j ? B : s - j;
                        if (b < 0.0 || pmem + (double)inflight * b * Aj * itp > c.mem) fm &= ~(1u << k);
                    }
                    lo = hi;
                }
                S.b2[r] = best;
                S.fmask[r] = (uint16_t)fm;
                S.bestk[r] = (uint16_t)bk;
            }
        }
        __syncthreads();
        // every B at once: each thread's least (bias, rank) among its groupings that fit
        double key[kMaxM];
        int idx[kMaxM];
#pragma unroll
        for (int k = 0; k < kMaxM; ++k) {
            key[k] = kInfP;
            idx[k] = 0x7fffffff;
        }
        for (int r = tid; r < nparts; r += kPxThreads) {
            const unsigned fm = S.fmask[r];
            const double v = S.b2[r];
#pragma unroll
            for (int k = 0; k < kMaxM; ++k)
                if (((fm >> k) & 1u) && (v < key[k] || (v == key[k] && r < idx[k]))) {
                    key[k] = v;
                    idx[k] = r;
                }
        }
        const int lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
#pragma unroll
        for (int k = 0; k < kMaxM; ++k) {
            if (k < A.n_m) {
                double kk = key[k];
                int ii = idx[k];
                wave_argmin(kk, ii);
                if (lane == 0) {
                    S.wkey[wv][k] = kk;
                    S.widx[wv][k] = ii;
                }
            }
        }
        __syncthreads();
        if (tid < A.n_m) {
            double kk = S.wkey[0][tid];
            int ii = S.widx[0][tid];
            for (int q = 1; q < kPxWaves; ++q) {
                const double ok = S.wkey[q][tid];
                const int oi = S.widx[q][tid];
                if (ok < kk || (ok == kk && oi < ii)) {
                    kk = ok;
                    ii = oi;
                }
            }
            S.minb2[tid] = kk;
            S.win[tid] = ii;
        }
        if (tid == 0) S.tiemask = 0u;
        __syncthreads();
        // another grouping with the same least bias: the least communication load decides
        for (int r = tid; r < nparts; r += kPxThreads) {
            const unsigned fm = S.fmask[r];
            const double v = S.b2[r];
            unsigned tb = 0u;
            for (int k = 0; k < A.n_m; ++k)
                if (((fm >> k) & 1u) && r != S.win[k] && v == S.minb2[k]) tb |= 1u << k;
            if (tb) atomicOr(&S.tiemask, tb);
        }
        __syncthreads();
        const unsigned ties = S.tiemask;
        for (int k = 0; k < A.n_m; ++k) {
            if (!((ties >> k) & 1u)) continue;
            const int B = S.mval[k];
            const double kb = S.minb2[k];
            double lk = kInfP;
            int li = 0x7fffffff;
            for (int r = tid; r < nparts; r += kPxThreads)
                if (((S.fmask[r] >> k) & 1u) && S.b2[r] == kb) {
                    const unsigned mask = unrank(r, c.O, s, S);
                    double D[16];
                    int q[16];
                    shares(mask, s, c.O, S, D, q);
                    const unsigned long long dexp = stage_exps(S.ms[S.bestk[r]], q, s);
                    unsigned long long texp;
                    double lc;
                    if (plan_lcomm(c, S, mask, s, B, dexp, texp, lc) && (lc < lk || (lc == lk && r < li))) {
                        lk = lc;
                        li = r;
                    }
                }
            block_argmin(lk, li, S);
            if (tid == 0) S.win[k] = li;
            __syncthreads();
        }
        // each B's proxy priced by its own thread
        if (tid < A.n_m && S.win[tid] != 0x7fffffff) {
            const int k = tid, B = S.mval[k], r = S.win[k];
            const unsigned mask = unrank(r, c.O, s, S);
            double D[16];
            int q[16];
            shares(mask, s, c.O, S, D, q);
            const unsigned long long dexp = stage_exps(S.ms[S.bestk[r]], q, s);
            unsigned long long texp;
            double lc;
            if (plan_lcomm(c, S, mask, s, B, dexp, texp, lc)) {
                S.gT[s][k] = price(c, S, mask, s, B, dexp, texp);
                S.gR[s][k] = r;
                S.gD[s][k] = dexp;
                S.gP[s][k] = texp;
            }
        }
        __syncthreads();   // S.ms is reloaded for the next degree
    }

    // the fastest grid; ties within the window: fewer stages, then fewer microbatches
    if (tid == 0) {
        double tmin = kInfP;
        for (int s = 1; s <= smax; ++s)
            for (int k = 0; k < A.n_m; ++k)
                if (S.gT[s][k] < tmin) tmin = S.gT[s][k];
        unsigned long long w0 = 0ull, w1 = 0ull, w2 = 0ull;
        float tout = __builtin_huge_valf(), thout = 0.0f;
        if (tmin < kInfP) {
            const double lim = tmin * (1.0 + A.tie_eps);
            int bs = 0, bk = -1;
            for (int s = 1; s <= smax && bk < 0; ++s) {
                for (int k = 0; k < A.n_m; ++k) {
                    if (!(S.gT[s][k] <= lim)) continue;
                    if (bk < 0 || S.mval[k] < S.mval[bk]) bk = k;
                }
                if (bk >= 0) bs = s;
            }
            const unsigned mask = unrank(S.gR[bs][bk], c.O, bs, S);
            const unsigned long long dexp = S.gD[bs][bk], texp = S.gP[bs][bk];
            const double T = S.gT[bs][bk];
            tout = (float)T;
            thout = (float)((double)c.Bg / T);
            w0 = (unsigned long long)(mask >> 1) | ((unsigned long long)bs << 16) |
                 ((unsigned long long)S.mval[bk] << 24) | (1ull << 31);
            w1 = dexp;
            w2 = texp;
        }
        A.t_iter[cell] = tout;
        A.thr[cell] = thout;
        A.plan[(size_t)cell * kProxyPlanWords + 0] = w0;
        A.plan[(size_t)cell * kProxyPlanWords + 1] = w1;
        A.plan[(size_t)cell * kProxyPlanWords + 2] = w2;
    }
}

// Resident blocks take cells from a device queue until none is left: a
// dispatcher that places block b on XCD b % 8 in order would otherwise leave
// CUs idle while a block waits for room on its XCD.
__global__ __launch_bounds__(kPxThreads) void proxy_kernel(ProxyArgs A, int n_cells)
{
    __shared__ ProxyLds S;
    __shared__ int slot;
    for (;;) {
        if (threadIdx.x == 0) {
            const unsigned long long q = atomicAdd(A.queue, 1ull);
            slot = q < (unsigned long long)n_cells ? (int)q : -1;
        }
        __syncthreads();
        const int cell = slot;
        __syncthreads();
        if (cell < 0) break;
        proxy_cell(A, S, cell);
        __syncthreads();          // the next cell reuses the LDS
    }
}

}  // namespace

hipError_t launch_proxy(const ProxyArgs& args, hipStream_t stream)
{
    const long long cells = (long long)args.n_jobs * args.n_types * args.n_counts;
    if (cells <= 0) return hipSuccess;
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, proxy_kernel, kPxThreads, 0);
    if (e != hipSuccess) return e;
    const long long resident = (long long)(args.n_cus > 0 ? args.n_cus : 1) * (per_cu > 0 ? per_cu : 1);
    const unsigned blocks = (unsigned)(cells < resident ? cells : resident);
    hipLaunchKernelGGL(proxy_kernel, dim3(blocks), dim3(kPxThreads), 0, stream, args, (int)cells);
    return hipGetLastError();
}

}  // namespace arena
