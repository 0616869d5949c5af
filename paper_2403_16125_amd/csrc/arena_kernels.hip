// HIP kernels of the plan-space estimator (gfx950 / CDNA4).
//
// A block of four 64-lane wavefronts owns one (job, GPU type) pair.
//   set-up   the job's layer tables, parameter/activation prefix sums and the
//            pure-compute cost prefix are staged in LDS once;
//   shared   stage-partition problems that do not depend on the GPU count
//            (the pure-compute problem, and every tensor degree when the
//            type has one contention factor for all counts) are solved once
//            per block for the union of the degrees any count requests;
//   cells    the waves then take GPU counts from an LDS work counter, solve
//            the count-specific problems, price every plan and reduce to the
//            cell's best plan.
// Nothing here is a dense contraction, so no MFMA: the work is compares,
// min/max and adds on the vector ALU; reductions use DPP row operations.
//
// Arithmetic is IEEE double.  The per-layer cost, its prefix sums, the
// balanced-partition value and the canonical cuts are evaluated in the same
// operation order as a plain left-to-right evaluation of the formulas in
// arena.h, so they are bit-reproducible; sums over stages are reduced in
// tree order.
#include <math.h>

#include "arena_internal.h"

namespace arena {
namespace {

constexpr double kInf = __builtin_huge_val();
constexpr int kSlotsShared = 10;   // 1 pure problem + up to 9 tensor-degree problems
constexpr int kPad = 8;            // prefix arrays hold +inf past the last layer
constexpr int kLevels = 7;         // successor tables: 2^7 > largest stage count - 1
constexpr int kLevelStride = 132;  // bytes per successor table (>= kLmax + 1)

struct WaveLds {
    double U[kLmax + kPad];       // cost prefix of the wave's current problem (+inf padded)
    double D[kLmax + kPad];       // partition recursion row, updated in place; while a plan is
                                  // priced, its bytes hold the successor tables of the cuts
    double Wt[kMaxTargets];       // bottleneck per requested degree (by rank)
    double planT[kMaxPlans];      // iteration time of each plan of the cell (+inf: does not fit)
    uint32_t planKey[kMaxPlans];  // pp << 12 | tp << 7 | m
    double bq[kMaxM];             // samples per microbatch of the admissible counts, ascending m
    int32_t mq[kMaxM];            // those microbatch counts
};
static_assert(kLevels * kLevelStride <= (int)sizeof(double) * (kLmax + kPad), "successor tables fit in D");

template <int SLOTS>
struct BlockLds {
    float t[kLmax];
    float x[kLmax];
    float q[kLmax];
    double Pp[kLmax + 1];         // prefix of parameter bytes
    double Ap[kLmax + 1];         // prefix of activation bytes
    double Upure[kLmax + kPad];   // prefix of the pure-compute per-sample cost (+inf padded)
    double Wtab[SLOTS][kLmax + 1];// bottleneck of each shared problem, by degree
    uint32_t adm[kMaxDp / 32];    // bit dp-1: some listed m has dp*m dividing the batch
    int32_t slot_tp[SLOTS];
    int32_t slot_var[SLOTS];
    int32_t n_slots;
    int32_t next_cell;
    int32_t uniform;              // one kappa for every count of this type
    int32_t moe;
    WaveLds w[kWavesPerBlock];
};

// ------------------------------------------------------------ wave helpers

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ double bcast(double v, int src)
{
    const unsigned long long b = (unsigned long long)__double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)(unsigned)(b & 0xffffffffull), src);
    const int hi = __builtin_amdgcn_readlane((int)(unsigned)(b >> 32), src);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) |
                                            (unsigned long long)(unsigned)lo));
}

template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp(double v, double ident)
{
    const unsigned long long b = (unsigned long long)__double_as_longlong(v);
    const unsigned long long e = (unsigned long long)__double_as_longlong(ident);
    const int lo = __builtin_amdgcn_update_dpp((int)(unsigned)e, (int)(unsigned)b, CTRL, ROWS, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(unsigned)(e >> 32), (int)(unsigned)(b >> 32), CTRL,
                                               ROWS, 0xf, false);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) |
                                            (unsigned long long)(unsigned)lo));
}

// Whole-wave reductions: quad swaps, row rotations, then row broadcasts leave
// the total in lane 63, which is broadcast (so every lane sees one value).
struct OpSum {
    static __device__ __forceinline__ double ident() { return 0.0; }
    static __device__ __forceinline__ double op(double a, double b) { return a + b; }
};
struct OpMax {
    static __device__ __forceinline__ double ident() { return -kInf; }
    static __device__ __forceinline__ double op(double a, double b) { return fmax(a, b); }
};
struct OpMin {
    static __device__ __forceinline__ double ident() { return kInf; }
    static __device__ __forceinline__ double op(double a, double b) { return fmin(a, b); }
};

template <class Op, int N>
__device__ __forceinline__ void wave_reduce(double (&v)[N])
{
    const double id = Op::ident();
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = Op::op(v[i], dpp<0xB1, 0xf>(v[i], id));   // quad_perm 1,0,3,2
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = Op::op(v[i], dpp<0x4E, 0xf>(v[i], id));   // quad_perm 2,3,0,1
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = Op::op(v[i], dpp<0x124, 0xf>(v[i], id));  // row_ror 4
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = Op::op(v[i], dpp<0x128, 0xf>(v[i], id));  // row_ror 8
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = Op::op(v[i], dpp<0x142, 0xa>(v[i], id));  // row_bcast 15
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = Op::op(v[i], dpp<0x143, 0xc>(v[i], id));  // row_bcast 31
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = bcast(v[i], 63);
}

template <class Op>
__device__ __forceinline__ double wave_reduce1(double x)
{
    double v[1] = {x};
    wave_reduce<Op, 1>(v);
    return v[0];
}

// Left-to-right prefix of L values held as (element lane, element lane+64):
// out[0] = 0, out[i] = out[i-1] + v[i-1].  Sequential on purpose: the rounding
// of a prefix must not depend on a reduction tree.  The values are staged in
// `tmp` (LDS) and one lane accumulates them in order: one add per layer.
// With `pad`, out[L+1 .. kLmax+kPad-1] = +inf (out has kLmax + kPad entries).
__device__ __forceinline__ void seq_prefix(double v0, double v1, int L, int lane, double* out, double* tmp,
                                           bool pad)
{
    if (lane < L) tmp[lane] = v0;
    if (lane + 64 < L) tmp[lane + 64] = v1;
    if (pad)
        for (int e = L + 1 + lane; e < kLmax + kPad; e += 64) out[e] = kInf;
    wave_sync();
    if (lane == 0) {
        double acc = 0.0;
        out[0] = 0.0;
#pragma unroll 8
        for (int i = 0; i < L; ++i) {
            acc = acc + tmp[i];
            out[i + 1] = acc;
        }
    }
    wave_sync();
}

// ------------------------------------------------------------ model pieces

struct JobCtx {
    int L, Bg;
    bool moe;       // has all-to-all layers
};

struct Cell {
    int n;          // GPUs of the cell
    double kappa;   // contention factor of the grid
    double B_pp;    // link between pipeline neighbours
    double c_p2p;   // kappa 2 / B_pp: p2p seconds per byte and sample, both directions
};

// Per-sample cost of each layer (formula in arena.h), prefix-summed into U.
__device__ void build_prefix_u(const float* t, const float* x, const float* q, double* U, double* tmp,
                               int lane, const JobCtx& jb, const TypeDev& ty, double kappa, int tp,
                               bool a2a_on)
{
    const double denom = (double)jb.Bg * ty.speed * (double)tp;
    const double ctp = kappa * 8.0 * (double)(tp - 1) / (double)tp;
    double u[2] = {0.0, 0.0};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int l = lane + 64 * s;
        if (l < jb.L) {
            double v = (double)t[l] / denom;
            if (tp > 1) v += ctp * (double)x[l] / ty.bw_intra;
            if (a2a_on) v += kappa * (double)q[l] / ty.bw_inter;
            u[s] = v;
        }
    }
    seq_prefix(u[0], u[1], jb.L, lane, U, tmp, true);
}

__device__ __forceinline__ bool adm_ok(const uint32_t* adm, int dp)
{
    return (adm[(dp - 1) >> 5] >> ((dp - 1) & 31)) & 1u;
}

// Is pp a requested degree of problem (n, tp, variant)?  pp divides n/tp, is
// at most the layer count, leaves an admissible data-parallel degree, and
// meets the all-to-all condition of the variant (variant 1: the MoE job's
// single-GPU-per-stage plan dp = tp = 1, which has no all-to-all).
__device__ __forceinline__ bool target_ok(const uint32_t* adm, const JobCtx& jb, int n, int tp,
                                          int variant, int pp)
{
    const int qn = n / tp;
    if (pp > jb.L || pp > qn || qn % pp != 0) return false;
    if (variant == 0) {
        if (jb.moe && pp >= n) return false;
    } else if (pp != n) {
        return false;
    }
    return adm_ok(adm, qn / pp);
}

// Degrees as a 128-bit mask (bit pp-1), uniform across the wave.
struct Mask {
    unsigned long long lo, hi;
    __device__ __forceinline__ bool test(int pp) const
    {
        return pp <= 64 ? ((lo >> (pp - 1)) & 1ull) : ((hi >> (pp - 65)) & 1ull);
    }
    __device__ __forceinline__ int count() const { return __popcll(lo) + __popcll(hi); }
    __device__ __forceinline__ int last() const
    {
        return hi ? 128 - __clzll(hi) : (lo ? 64 - __clzll(lo) : 0);
    }
    // smallest set degree >= from (0 if none)
    __device__ __forceinline__ int next(int from) const
    {
        if (from <= 64) {
            const unsigned long long m = from <= 1 ? lo : (lo & ~((1ull << (from - 1)) - 1ull));
            if (m) return __ffsll((long long)m);
            return hi ? 64 + __ffsll((long long)hi) : 0;
        }
        if (from > 128) return 0;
        const unsigned long long m = hi & ~((1ull << (from - 65)) - 1ull);
        return m ? 64 + __ffsll((long long)m) : 0;
    }
};

__device__ __forceinline__ Mask ballot_mask(bool ok0, bool ok1)
{
    Mask m;
    m.lo = __ballot(ok0);
    m.hi = __ballot(ok1);
    return m;
}

// ------------------------------------------------------------ partition

// DPP lane shift: lane l receives lane l+1's value (lane 63 keeps `last`).
__device__ __forceinline__ int from_next_lane(int v, int last)
{
    return __builtin_amdgcn_update_dpp(last, v, 0x130, 0xf, 0xf, false);   // wave_shl:1
}

// One lane of row k of the recursion D_k(i) = min_j max(D_{k-1}(j), U_i - U_j)
// (D holds row k-1 and receives row k in place).  The crossing c -- the first
// j >= k-1 with D_{k-1}(j) >= U_i - U_j -- never moves left as i or k grows,
// so it is at least the crossing this lane found for i-1 and the one the next
// lane found for i in row k-1 (`lb`).  Position i always passes the test: D[i]
// holds D_{k-1}(i) >= 0 = U_i - U_i, or +inf where row k-1 stopped short of i,
// so the first passing position of a probe is c whenever the probe reaches i
// and nothing to the right of i is ever looked at.  Four candidates are tested
// in one round of loads; farther crossings gallop and then bisect.
//   D_k(i) = min(D_{k-1}(c), U_i - U_{c-1})   (second term only for c-1 >= k-1)
// At c = i the first term is D_{k-1}(i) >= U_i - U_{i-1} (every partition of
// the first i layers has a stage holding layer i-1 whole) or +inf, so the
// minimum is U_i - U_{i-1}, the value of the only split left.
__device__ __forceinline__ void dp_entry(const double* U, double* D, int k, int hi, int i, int lb, int& jp)
{
    const bool act = i <= hi;
    double v = 0.0;
    if (act) {
        const double Ui = U[i];
        const int a = lb > k - 1 ? lb : k - 1;   // every j < a fails
        const bool f0 = D[a] >= Ui - U[a];
        const bool f1 = D[a + 1] >= Ui - U[a + 1];
        const bool f2 = D[a + 2] >= Ui - U[a + 2];
        const bool f3 = D[a + 3] >= Ui - U[a + 3];
        int c = f0 ? a : f1 ? a + 1 : f2 ? a + 2 : a + 3;
        if (!(f0 | f1 | f2 | f3)) {
            // rare: crossing in (a+3, i]; i passes without a look
            int lo = a + 4, b = i, step = 1;
            while (lo < b) {
                int p = lo + step - 1;
                p = p < b - 1 ? p : b - 1;
                if (D[p] >= Ui - U[p]) { b = p; break; }
                lo = p + 1;
                step <<= 1;
            }
            while (lo < b) {
                const int mid = (lo + b) >> 1;
                if (D[mid] >= Ui - U[mid]) b = mid; else lo = mid + 1;
            }
            c = lo;
        }
        jp = c;
        const double dc = D[c];
        const double t = Ui - U[c - 1];
        v = (c >= k && t < dc) ? t : dc;
    }
    // every lane has read row k-1 before any lane overwrites it
    __asm__ volatile("" ::: "memory");
    if (act) D[i] = v;
}

// Bottleneck W*(pp) for every degree in `tm`, written to Wout[pp] (by_pp) or
// Wout[rank of pp].  Row k is evaluated for i in [k, L - tau(k) + k] only,
// tau(k) the smallest requested degree >= k: larger i cannot reach a
// requested cell.  Lane l of row k takes i = k + l (+64): the window width
// never grows with k, so after the first rows one pass covers a row, and a
// lane's crossing from row k-1 (for i-1) is a lower bound for row k.  After
// each row, D[hi+1] = +inf marks the first position the row did not reach.
__device__ void solve_dp(const double* U, double* D, int L, const Mask& tm, double* Wout, bool by_pp,
                         int lane, unsigned long long& entries)
{
    const int P = tm.last();
    int tau = tm.next(1);
    int rank = 0;
    unsigned n_ent = 0;
    {
        const int hi = L - tau + 1;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int i = 1 + lane + 64 * s;
            if (i <= hi) D[i] = U[i];
        }
        if (lane == 0) D[hi + 1] = kInf;
        n_ent += (unsigned)hi;
        wave_sync();
        if (tau == 1) {
            if (lane == 0) Wout[by_pp ? 1 : 0] = D[L];
            ++rank;
            tau = tm.next(2);
        }
    }
    int jp0 = 0, jp1 = 0;
    for (int k = 2; k <= P; ++k) {
        const int hi = L - tau + k;
        // lower bounds: own crossing (i-1, row k-1) and the next lane's (i, row k-1)
        const int top1 = __builtin_amdgcn_readlane(jp1, 0);
        const int nb0 = from_next_lane(jp0, top1);
        const int nb1 = from_next_lane(jp1, jp1);
        const int lb0 = jp0 > nb0 ? jp0 : nb0;
        const int lb1 = jp1 > nb1 ? jp1 : nb1;
        if (hi - k >= 64) dp_entry(U, D, k, hi, k + 64 + lane, lb1, jp1);   // high part first: in place
        dp_entry(U, D, k, hi, k + lane, lb0, jp0);
        if (lane == 0) D[hi + 1] = kInf;
        n_ent += (unsigned)(hi - k + 1);
        wave_sync();
        if (k == tau) {
            if (lane == 0) Wout[by_pp ? k : rank] = D[L];
            ++rank;
            tau = tm.next(k + 1);
        }
    }
    entries += n_ent;
    wave_sync();
}

// Canonical cuts for degree pp and bottleneck W: c_pp = L and, right to left,
// c_k = max(k, next(c_{k+1})) with next(e) the smallest c such that
// U_e - U_c <= W.  Unrolled: next(e) < e, so a_k = next^(pp-k)(L) falls by at
// least one per step and a_k - k never decreases as k falls; once the clamp
// bites it bites for every smaller k, hence c_k = max(k, a_k).  Every lane
// finds next(e) for its layers by binary lifting over U, the wave builds the
// successor tables next^(2^s) in LDS bytes `J` (level s at J + s kLevelStride,
// node 0 maps to itself) and lane k walks pp-k steps from L in log2 jumps.
// Returns the bounds of stage s = lane + 64h as [lo_h, hi_h) = [c_s, c_{s+1}).
struct Stages {
    int lo0, lo1, hi0, hi1;
};

__device__ Stages canonical_stages(const double* U, uint8_t* J, int lane, int L, int pp, double W)
{
    Stages r;
    if (pp == 1) {
        r.lo0 = 0; r.hi0 = L; r.lo1 = 0; r.hi1 = 0;
        return r;
    }
    const int levels = 32 - __clz(pp - 1);   // 2^levels > pp - 1
    // next(e): the failing c (U_e - U_c > W) form a prefix of [0, e); c = e-1
    // passes (W is at least every single-layer cost) and so does every c > e-1
    // (U is non-decreasing and +inf past L)
    int cur0 = 0, cur1 = 0;
    const int e0 = 1 + lane, e1 = 65 + lane;
    if (e0 <= L) {
        const double Ue = U[e0];
        int pos = 0;
#pragma unroll
        for (int step = 32; step >= 1; step >>= 1)
            if (Ue - U[pos + step - 1] > W) pos += step;
        cur0 = pos;
        J[e0] = (uint8_t)pos;
    }
    if (L > 64 && e1 <= L) {
        const double Ue = U[e1];
        int pos = 0;
#pragma unroll
        for (int step = 64; step >= 1; step >>= 1)
            if (Ue - U[pos + step - 1] > W) pos += step;
        cur1 = pos;
        J[e1] = (uint8_t)pos;
    }
    if (lane < levels) J[lane * kLevelStride] = 0;
    wave_sync();
    for (int s = 1; s < levels; ++s) {
        const uint8_t* prev = J + (s - 1) * kLevelStride;
        uint8_t* lev = J + s * kLevelStride;
        if (e0 <= L) cur0 = prev[cur0];
        if (L > 64 && e1 <= L) cur1 = prev[cur1];
        if (e0 <= L) lev[e0] = (uint8_t)cur0;
        if (L > 64 && e1 <= L) lev[e1] = (uint8_t)cur1;
        wave_sync();
    }
    // c_k for k = lane (cA) and k = lane + 64 (cB); c_0 = 0, c_pp = L
    int cA = 0, cB = 0;
    {
        const int k = lane;
        if (k >= 1 && k < pp) {
            const int d = pp - k;
            int node = L;
            for (int s = 0; s < levels; ++s) {
                const int nd = J[s * kLevelStride + node];
                node = ((d >> s) & 1) ? nd : node;
            }
            cA = node > k ? node : k;
        }
        cA = k == pp ? L : cA;
    }
    if (pp >= 64) {
        const int k = lane + 64;
        if (k < pp) {
            const int d = pp - k;
            int node = L;
            for (int s = 0; s < levels; ++s) {
                const int nd = J[s * kLevelStride + node];
                node = ((d >> s) & 1) ? nd : node;
            }
            cB = node > k ? node : k;
        }
        cB = k == pp ? L : cB;
    }
    // stage s ends where stage s+1 starts: the next lane's cut (lane 63 of the
    // low half takes c_64, lane 63 of the high half c_128)
    r.lo0 = cA;
    r.hi0 = from_next_lane(cA, __builtin_amdgcn_readlane(cB, 0));
    r.lo1 = cB;
    r.hi1 = from_next_lane(cB, pp == 128 ? L : 0);
    return r;
}

// Price every admissible microbatch count of plan (dp, tp, pp) with the
// canonical stages of bottleneck W; appends to the wave's plan buffer.  Lane
// mi < n_m holds m_values[mi] (ascending) in `mv`: the lanes price one count
// each.  A stage's memory is non-increasing in m (min(m, pp-k) b is the batch
// share Bg/dp while m <= pp-k and falls after), so the counts that fit are the
// top of the admissible list; the first one is found by bisection.
template <int SLOTS>
__device__ void price_target(const BlockLds<SLOTS>& B, WaveLds& Wv, const double* U, int lane, int mv,
                             const JobCtx& jb, const TypeDev& ty, const Cell& cell, int tp, int pp,
                             double W, int& np, unsigned long long& overflow)
{
    const Stages sg = canonical_stages(U, reinterpret_cast<uint8_t*>(Wv.D), lane, jb.L, pp, W);
    const int dp = cell.n / (tp * pp);
    const int grp = dp * tp;
    const double B_dp = (grp <= ty.gpn && ty.gpn % grp == 0) ? ty.bw_intra : ty.bw_inter;

    // per-stage parameter and activation bytes of the lane's stages
    const bool act0 = lane < pp, act1 = lane + 64 < pp;
    double P0 = 0.0, A0 = 0.0, P1 = 0.0, A1 = 0.0, sx = 0.0;
    if (act0) {
        P0 = B.Pp[sg.hi0] - B.Pp[sg.lo0];
        A0 = B.Ap[sg.hi0] - B.Ap[sg.lo0];
        if (lane < pp - 1) sx = (double)B.x[sg.hi0 - 1];
    }
    if (act1) {
        P1 = B.Pp[sg.hi1] - B.Pp[sg.lo1];
        A1 = B.Ap[sg.hi1] - B.Ap[sg.lo1];
        if (lane + 64 < pp - 1) sx += (double)B.x[sg.hi1 - 1];
    }
    double rs[1] = {sx}, rm[1] = {fmax(P0, P1)};
    wave_reduce<OpSum, 1>(rs);
    wave_reduce<OpMax, 1>(rm);
    const double sumX = rs[0];
    const double pmax = rm[0];
    const double sumS = U[jb.L];   // the stages tile the layers: sum of stage costs
    const double ar = (dp > 1)
        ? pmax * (cell.kappa * 2.0 * (double)(dp - 1) / ((double)dp * (double)tp * B_dp))
        : 0.0;
    const double per_sample = sumS + cell.c_p2p * sumX;   // fill time per sample

    // lanes over the microbatch counts: admissible when dp m divides the batch
    // (the quotient of a correctly rounded division is exact then)
    bool adm = false;
    double b = 0.0;
    if (mv > 0) {
        const double dm = (double)(dp * mv);
        const double q = rint((double)jb.Bg / dm);
        adm = q * dm == (double)jb.Bg;
        b = q;
    }
    const unsigned long long amask = __ballot(adm);
    const int nadm = __popcll(amask);
    if (nadm == 0) return;
    const int rank = __builtin_amdgcn_mbcnt_hi((unsigned)(amask >> 32),
                                               __builtin_amdgcn_mbcnt_lo((unsigned)amask, 0u));
    if (adm) {
        Wv.bq[rank] = b;
        Wv.mq[rank] = mv;
    }
    wave_sync();

    // memory: 4 P_k + min(m, pp-k) b A_k <= mem tp on every stage
    const double cap = ty.mem * (double)tp;
    const double fP0 = 4.0 * P0, fP1 = 4.0 * P1;
    const int r0 = pp - lane, r1 = pp - lane - 64;         // stages from the lane's to the last
    int lo = 0, hi = nadm;                                  // first fitting rank in [lo, hi]
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        const double bm = Wv.bq[mid];
        const int m = Wv.mq[mid];
        const double i0 = (double)(m < r0 ? m : r0) * bm;
        const double i1 = (double)(m < r1 ? m : r1) * bm;
        const bool over = (act0 && fP0 + i0 * A0 > cap) || (act1 && fP1 + i1 * A1 > cap);
        if (__ballot(over) == 0ull) hi = mid; else lo = mid + 1;
    }

    if (adm) {
        const double T = b * per_sample + (double)(mv - 1) * (b * W) + ar;
        const int slot = np + rank;
        if (slot < kMaxPlans) {
            Wv.planT[slot] = rank >= lo ? T : kInf;
            Wv.planKey[slot] = ((unsigned)pp << 12) | ((unsigned)tp << 7) | (unsigned)mv;
        }
    }
    np += nadm;
    if (np > kMaxPlans) {
        overflow = 1;
        np = kMaxPlans;
    }
}

// ------------------------------------------------------------ the kernel

template <int SLOTS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void estimate_kernel(EstimateArgs A)
{
    __shared__ BlockLds<SLOTS> B;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    WaveLds& Wv = B.w[wid];

    const int item = A.item_order[blockIdx.x];
    const int j = item / A.n_types;
    const int g = item - j * A.n_types;
    const int off = A.layer_offset[j];
    JobCtx jb;
    jb.L = A.layer_offset[j + 1] - off;
    jb.Bg = A.batch[j];
    const TypeDev ty = A.types[g];
    int mv = 0;                      // lane mi: the mi-th microbatch count (ascending), 0 past the list
#pragma unroll
    for (int i = 0; i < kMaxM; ++i)
        if (lane == i && i < A.n_m) mv = A.m_values[i];

    // ---- stage the job
    bool has_q = false;
    if (tid < jb.L) {
        B.t[tid] = A.t[off + tid];
        B.x[tid] = A.x[off + tid];
        const float qv = A.q[off + tid];
        B.q[tid] = qv;
        has_q = qv > 0.0f;
    }
    jb.moe = __syncthreads_or(has_q) != 0;
    if (wid == 0 || wid == 1) {
        const float* src = (wid == 0 ? A.p : A.a) + off;
        const double v0 = lane < jb.L ? (double)src[lane] : 0.0;
        const double v1 = lane + 64 < jb.L ? (double)src[lane + 64] : 0.0;
        seq_prefix(v0, v1, jb.L, lane, wid == 0 ? B.Pp : B.Ap, Wv.D, false);
    } else if (wid == 2) {
        build_prefix_u(B.t, B.x, B.q, B.Upure, Wv.D, lane, jb, ty, 1.0, 1, false);
    } else {
        bool same = true;
        for (int c = lane; c < A.n_counts; c += 64) same &= A.kappa[g * A.n_counts + c] == A.kappa[g * A.n_counts];
        const bool uni = __ballot(!same) == 0ull;
        if (lane == 0) {
            B.uniform = uni ? 1 : 0;
            B.next_cell = 0;
            B.moe = jb.moe ? 1 : 0;
        }
    }
    // admissible data-parallel degrees: dp*m divides the batch for a listed m
    for (int base = 0; base < kMaxDp; base += 256) {
        const int dp = base + tid + 1;
        bool ok = false;
        for (int i = 0; i < A.n_m; ++i) ok |= (jb.Bg % (dp * A.m_values[i])) == 0;
        const unsigned long long bits = __ballot(ok);
        if (lane == 0) {
            B.adm[(base + 64 * wid) >> 5] = (uint32_t)(bits & 0xffffffffull);
            B.adm[((base + 64 * wid) >> 5) + 1] = (uint32_t)(bits >> 32);
        }
    }
    __syncthreads();

    // ---- shared problems: the pure-compute one, and every tensor degree when
    // the type's contention factor is the same for all counts
    if (tid == 0) {
        int ns = 0;
        B.slot_tp[ns] = 1;
        B.slot_var[ns] = jb.moe ? 1 : 0;
        ++ns;
        if (SLOTS > 1 && A.share_tp && B.uniform) {
            for (int tp = 1; tp <= ty.gpn && ns < SLOTS; ++tp) {
                if (ty.gpn % tp != 0 || (tp == 1 && !jb.moe)) continue;
                B.slot_tp[ns] = tp;
                B.slot_var[ns] = 0;
                ++ns;
            }
        }
        B.n_slots = ns;
    }
    __syncthreads();
    const int n_slots = B.n_slots;

    unsigned long long n_plans = 0, n_problems = 0, dp_entries = 0, n_infeasible = 0, overflow = 0;

    for (int s = wid; s < n_slots; s += kWavesPerBlock) {
        const int tp = B.slot_tp[s], var = B.slot_var[s];
        bool ok0 = false, ok1 = false;
        for (int c = 0; c < A.n_counts; ++c) {
            const int n = A.counts[c];
            if (n % tp != 0) continue;
            ok0 |= target_ok(B.adm, jb, n, tp, var, 1 + lane);
            ok1 |= target_ok(B.adm, jb, n, tp, var, 65 + lane);
        }
        const Mask tm = ballot_mask(ok0, ok1);
        if (tm.count() == 0) continue;
        const double* U = B.Upure;
        if (s > 0) {
            build_prefix_u(B.t, B.x, B.q, Wv.U, Wv.D, lane, jb, ty, (double)A.kappa[g * A.n_counts], tp,
                           true);
            U = Wv.U;
        }
        solve_dp(U, Wv.D, jb.L, tm, B.Wtab[s], true, lane, dp_entries);
        ++n_problems;
    }
    __syncthreads();

    // ---- cells: take counts, largest first, from the block's work counter
    for (;;) {
        int cix = 0;
        if (lane == 0) cix = atomicAdd(&B.next_cell, 1);
        cix = __builtin_amdgcn_readfirstlane(cix);
        if (cix >= A.n_counts) break;
        const int ci = A.count_order[cix];
        Cell cell;
        cell.n = A.counts[ci];
        cell.kappa = (double)A.kappa[g * A.n_counts + ci];
        cell.B_pp = (cell.n <= ty.gpn) ? ty.bw_intra : ty.bw_inter;
        cell.c_p2p = cell.kappa * 2.0 / cell.B_pp;
        int np = 0;

        const int tpmax = cell.n < ty.gpn ? cell.n : ty.gpn;
        for (int tp = 1; tp <= tpmax; ++tp) {
            if (cell.n % tp != 0 || ty.gpn % tp != 0) continue;
            for (int var = 0; var < 2; ++var) {
                if (var == 1 && !(jb.moe && tp == 1)) break;
                const Mask tm = ballot_mask(target_ok(B.adm, jb, cell.n, tp, var, 1 + lane),
                                            target_ok(B.adm, jb, cell.n, tp, var, 65 + lane));
                if (tm.count() == 0) continue;
                // shared problem?
                int slot = -1;
                if (tp == 1 && (var == 1 || !jb.moe)) slot = 0;
                else
                    for (int s = 1; s < n_slots; ++s)
                        if (B.slot_tp[s] == tp && B.slot_var[s] == var) slot = s;
                const double* U;
                if (slot == 0) {
                    U = B.Upure;
                } else {
                    build_prefix_u(B.t, B.x, B.q, Wv.U, Wv.D, lane, jb, ty, cell.kappa, tp, var == 0);
                    U = Wv.U;
                }
                if (slot < 0) {
                    solve_dp(U, Wv.D, jb.L, tm, Wv.Wt, false, lane, dp_entries);
                    ++n_problems;
                }
                int rank = 0;
                for (int pp = tm.next(1); pp; pp = tm.next(pp + 1), ++rank) {
                    const double W = slot >= 0 ? B.Wtab[slot][pp] : Wv.Wt[rank];
                    price_target(B, Wv, U, lane, mv, jb, ty, cell, tp, pp, W, np, overflow);
                }
            }
        }
        wave_sync();

        // best plan of the cell: smallest key among plans within the tie window
        double tl = kInf;
        for (int e = lane; e < np; e += 64) tl = fmin(tl, Wv.planT[e]);
        const double tmin = wave_reduce1<OpMin>(tl);
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
            wave_sync();
            continue;
        }
        const double lim = tmin * (1.0 + A.tie_eps);
        double kl = kInf;
        for (int e = lane; e < np; e += 64)
            if (Wv.planT[e] <= lim) kl = fmin(kl, (double)Wv.planKey[e]);
        const unsigned kbest = (unsigned)wave_reduce1<OpMin>(kl);
        double il = -1.0;
        for (int e = lane; e < np; e += 64)
            if (Wv.planKey[e] == kbest) il = (double)e;
        int ib = (int)wave_reduce1<OpMax>(il);
        ib = ib < 0 ? 0 : (ib >= np ? np - 1 : ib);
        const double Tb = Wv.planT[ib];
        const int pp = (int)(kbest >> 12);
        const int tp = (int)((kbest >> 7) & 0x1Fu);
        const int m = (int)(kbest & 0x7Fu);
        const int dp = cell.n / (tp * pp);
        if (lane == 0) {
            A.t_iter[cidx] = (float)Tb;
            A.thr[cidx] = (float)((double)jb.Bg / Tb);
            A.plan[cidx] = (unsigned)dp | ((unsigned)tp << 11) | ((unsigned)pp << 16) |
                           ((unsigned)m << 24) | (1u << 31);
        }
        if (A.cuts) {
            // re-derive the winner's bottleneck and cuts
            const int var = (jb.moe && dp * tp == 1) ? 1 : 0;
            int slot = -1;
            if (tp == 1 && (var == 1 || !jb.moe)) slot = 0;
            else
                for (int s = 1; s < n_slots; ++s)
                    if (B.slot_tp[s] == tp && B.slot_var[s] == var) slot = s;
            const double* U;
            if (slot == 0) {
                U = B.Upure;
            } else {
                build_prefix_u(B.t, B.x, B.q, Wv.U, Wv.D, lane, jb, ty, cell.kappa, tp, var == 0);
                U = Wv.U;
            }
            double W;
            if (slot >= 0) {
                W = B.Wtab[slot][pp];
            } else {
                Mask one;
                one.lo = pp <= 64 ? (1ull << (pp - 1)) : 0ull;
                one.hi = pp > 64 ? (1ull << (pp - 65)) : 0ull;
                unsigned long long scratch_entries = 0;
                solve_dp(U, Wv.D, jb.L, one, Wv.Wt, false, lane, scratch_entries);
                W = Wv.Wt[0];
            }
            const Stages sg = canonical_stages(U, reinterpret_cast<uint8_t*>(Wv.D), lane, jb.L, pp, W);
            uint8_t* row = A.cuts + cidx * A.cuts_stride;
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const int idx = lane + 64 * s;
                const int en = s == 0 ? sg.hi0 : sg.hi1;
                if (idx < A.cuts_stride) row[idx] = (idx < pp - 1) ? (uint8_t)en : (uint8_t)0xFF;
            }
            for (int e = 128 + lane; e < A.cuts_stride; e += 64) row[e] = 0xFF;
        }
        wave_sync();
    }

    if (lane == 0) {
        if (wid == 0) atomicAdd(&A.counters[kCells], (unsigned long long)A.n_counts);
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
    if (args.share_tp)
        hipLaunchKernelGGL(estimate_kernel<kSlotsShared>, dim3((unsigned)blocks), dim3(256), 0, stream, args);
    else
        hipLaunchKernelGGL(estimate_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, stream, args);
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
