// HIP kernels of the plan-space estimator (gfx950 / CDNA4).
//
// A block of four 64-lane wavefronts works on one (job, GPU type) pair at a
// time; one block per resident slot is launched and each takes pairs from a
// device queue, heaviest first, until none is left.
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

#include <mutex>

#include "arena_internal.h"

namespace arena {
namespace {

constexpr double kInf = __builtin_huge_val();
constexpr int kSlotsShared = 10;   // 1 pure problem + up to 9 tensor-degree problems
constexpr int kPad = 8;            // prefix arrays hold +inf past the last layer
constexpr int kLevels = 7;         // successor tables: 2^7 > largest stage count - 1
constexpr int kLevelStride = 132;  // bytes per successor table (>= kLmax + 1)
constexpr int kMaxCand = 8;        // tensor degrees of one cell (divisors of a node size <= 31)
static_assert(kMaxPlans <= 256, "plan entries are packed below the key in 8 bits");
constexpr int kCertMinDegree = 2;  // a bottleneck certificate is tried for degrees from here up
constexpr int kHeadLayers = 2;     // leading layers whose own memory bounds every plan (lower bounds)
constexpr int kCertRounds = 3;     // splits tried per certificate (2 under the memory rule, whose
                                   // pricing order they change to its cost)

struct WaveLds {
    // the wave's current problem, pairs (U_j, D_j): U the cost prefix (+inf
    // padded), D the partition recursion row, updated in place
    alignas(16) double UD[2 * (kLmax + kPad)];
    double planT[kMaxPlans];      // iteration time of each plan of the cell (+inf: does not fit)
    uint32_t planKey[kMaxPlans];  // pp << 12 | tp << 7 | m
    double bq[kMaxM];             // samples per microbatch of the admissible counts, ascending m
    int32_t mq[kMaxM];            // those microbatch counts
    double lbnd[kLmax];           // lower bound of the iteration time, by pipeline degree - 1
    uint8_t tq[64];               // a problem's requested degrees, compacted
    double cand_lb[kMaxCand];     // the cell's tensor-degree problems: least lower bound of their plans
    uint8_t cand_tp[kMaxCand];    //   and their tensor degree
    uint8_t cutrow[kLmax];        // with cuts on: the cut row of the plan holding the best time
    double cut_T;                 //   that time (+inf: none yet)
    int32_t cut_tp, cut_pp;       //   and its degrees
    int32_t cut_m;                //   memory rule: its m if the row fits only under the rule, else 0
    int32_t cut_mfit;             //   the smallest m the balanced row fits
    unsigned long long tally[kNumCounters];   // the wave's work tallies (lane 0 updates)
    union {
        uint8_t J[kLevels * kLevelStride];   // successor tables of the canonical cuts
        double R[kLmax + 1];                 // memory rule: its recursion row (never live with J)
    };
};

template <int SLOTS>
struct BlockLds {
    float t[kLmax];
    float x[kLmax];
    float q[kLmax];
    double Pp[kLmax + 1];         // prefix of parameter bytes
    double Ap[kLmax + 1];         // prefix of activation bytes
    double Upure[kLmax + kPad];   // prefix of the pure-compute per-sample cost (+inf padded)
    double Wtab[SLOTS][kLmax + 1];// bottleneck of each shared problem, by degree (slot 0, the
                                  // pure-compute problem: every degree up to the layer count)
    uint8_t mmax[kMaxDp];         // [dp-1]: largest listed m with dp*m dividing the batch, 0: none
    uint8_t mcnt[kMaxDp];         // [dp-1]: how many listed m have dp*m dividing the batch
    double p_layer_max;           // largest parameter bytes of one layer
    double x_layer_min;           // smallest boundary activation bytes of one layer
    double x_sum, q_sum;          // sums over the layers of x and of the all-to-all bytes
    double head_p[kHeadLayers];   // parameter and activation bytes of the leading layers, as prefix
    double head_a[kHeadLayers];   //   differences (0 past the layer count)
    float xwin[kLmax + 1];        // [pp]: least x bytes of a window of layers whose pure-compute cost
    float qwin[kLmax + 1];        //   reaches Wtab[0][pp], and least all-to-all bytes (rounded down)
    int32_t slot_tp[SLOTS];
    int32_t slot_var[SLOTS];
    int32_t n_slots;
    int32_t next_cell;
    int32_t uniform;              // one kappa for every count of this type
    int32_t moe;
    unsigned long long pure_cached[2];   // bit pp-1: the block's cache row of the pure split of pp is current
    WaveLds w[kWavesPerBlock];
};

// ------------------------------------------------------------ wave helpers

// Orders the LDS accesses of the lanes of one wave: its memory operations
// execute in order, so wavefront-scope fences only stop the compiler from
// moving accesses across (no wait for completion).
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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
// Element e of out (tmp) sits at out[e * OS] (tmp[e * TS]).
template <int OS, int TS>
__device__ __forceinline__ void seq_prefix(double v0, double v1, int L, int lane, double* out, double* tmp,
                                           bool pad)
{
    if (lane < L) tmp[lane * TS] = v0;
    if (lane + 64 < L) tmp[(lane + 64) * TS] = v1;
    if (pad)
        for (int e = L + 1 + lane; e < kLmax + kPad; e += 64) out[e * OS] = kInf;
    wave_sync();
    if (lane == 0) {
        double acc = 0.0;
        out[0] = 0.0;
        // eight loads issued before their adds and stores (a store may alias a
        // later load, so the compiler would otherwise wait on each load in turn)
        int i = 0;
        for (; i + 8 <= L; i += 8) {
            double v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = tmp[(i + k) * TS];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                acc = acc + v[k];
                out[(i + k + 1) * OS] = acc;
            }
        }
        for (; i < L; ++i) {
            acc = acc + tmp[i * TS];
            out[(i + 1) * OS] = acc;
        }
    }
    wave_sync();
}

// Adds a wave-uniform amount to one of the wave's tallies.
__device__ __forceinline__ void tally(WaveLds& Wv, int lane, int which, unsigned long long v)
{
    if (lane == 0) Wv.tally[which] += v;
}

// 1/x to within a few ulps: the hardware estimate refined by one Newton step
// (lower bounds use it under a margin of 1e-9; integer quotients rounded from
// it are exact when the division is).
__device__ __forceinline__ double rcp_approx(double x)
{
    const double r = __builtin_amdgcn_rcp(x);
    return fma(fma(-x, r, 1.0), r, r);
}

// ------------------------------------------------------------ model pieces

// Does a group of grp GPUs (>= 1) tile a node (grp divides the node size)?
__device__ __forceinline__ bool tiles_node(const TypeDev& ty, int grp)
{
    return grp < 32 && ((ty.divs >> grp) & 1u);
}

// n / d for d dividing n <= ARENA_MAX_GPU_COUNT: the float quotient is
// within 1e-6 relative of the integer, which rounding recovers.
__device__ __forceinline__ int exact_quot(int n, int d)
{
    return (int)rintf((float)n * __builtin_amdgcn_rcpf((float)d));
}

// Link bandwidth by value (a conditional over two fields of one struct would
// select an address and keep the struct in private memory).
__device__ __forceinline__ double link_bw(bool intra, const TypeDev& ty)
{
    const double a = ty.bw_intra;
    const double b = ty.bw_inter;
    return intra ? a : b;
}

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

// Per-sample cost of layers lane and lane+64 (formula in arena.h; 0 past L).
__device__ __forceinline__ void layer_costs(const float* t, const float* x, const float* q, int lane,
                                            const JobCtx& jb, const TypeDev& ty, double kappa, int tp,
                                            bool a2a_on, double (&u)[2])
{
    const double denom = (double)jb.Bg * ty.speed * (double)tp;
    const double ctp = kappa * 8.0 * (double)(tp - 1) / (double)tp;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int l = lane + 64 * s;
        u[s] = 0.0;
        if (l < jb.L) {
            double v = (double)t[l] / denom;
            if (tp > 1) v += ctp * (double)x[l] / ty.bw_intra;
            if (a2a_on) v += kappa * (double)q[l] / ty.bw_inter;
            u[s] = v;
        }
    }
}

// Per-sample cost of each layer, prefix-summed into U (+inf past L; element
// e at U[e * OS]), staged in tmp (element e at tmp[2 e]).
template <int OS>
__device__ void build_prefix_u(const float* t, const float* x, const float* q, double* U, double* tmp,
                               int lane, const JobCtx& jb, const TypeDev& ty, double kappa, int tp,
                               bool a2a_on)
{
    double u[2];
    layer_costs(t, x, q, lane, jb, ty, kappa, tp, a2a_on, u);
    seq_prefix<OS, 2>(u[0], u[1], jb.L, lane, U, tmp, true);
}

__device__ __forceinline__ bool adm_ok(const uint8_t* mmax, int dp)
{
    return mmax[dp - 1] != 0;
}

// Is pp a requested degree of problem (n, tp, variant), tp dividing n?  pp divides n/tp, is
// at most the layer count, leaves an admissible data-parallel degree, and
// meets the all-to-all condition of the variant (variant 1: the MoE job's
// single-GPU-per-stage plan dp = tp = 1, which has no all-to-all).
__device__ __forceinline__ bool target_ok(const uint8_t* adm, const JobCtx& jb, int n, int tp,
                                          int variant, int pp)
{
    const int qn = exact_quot(n, tp);
    if (pp > jb.L || pp > qn) return false;
    // qn / pp when pp divides qn (qn <= 1024: the float quotient is within 1e-3)
    const int d = (int)rintf((float)qn * __builtin_amdgcn_rcpf((float)pp));
    if (__umul24(d, pp) != qn) return false;
    if (variant == 0) {
        if (jb.moe && pp >= n) return false;
    } else if (pp != n) {
        return false;
    }
    return adm_ok(adm, d);
}

// Degrees as a 128-bit mask (bit pp-1), uniform across the wave.
struct Mask {
    unsigned long long lo, hi;
    __device__ __forceinline__ bool test(int pp) const
    {
        return pp <= 64 ? ((lo >> (pp - 1)) & 1ull) : ((hi >> (pp - 65)) & 1ull);
    }
    __device__ __forceinline__ int count() const { return __popcll(lo) + __popcll(hi); }
    __device__ __forceinline__ bool any() const { return (lo | hi) != 0ull; }
    __device__ __forceinline__ Mask operator&(const Mask& o) const { return Mask{lo & o.lo, hi & o.hi}; }
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
__device__ __forceinline__ void dp_entry(double* UD, int k, int hi, int i, int lb, int& jp)
{
    // U_j = UD[2j], D_j = UD[2j+1]
    const bool act = i <= hi;
    double v;                                // set and stored only where act
    if (act) {
        const double Ui = UD[2 * i];
        const int a = lb > k - 1 ? lb : k - 1;   // every j < a fails
        const double* P = UD + 2 * a;
        // two candidates for every lane, two more only where neither passed
        // (an inactive lane moves no LDS data)
        const bool f0 = P[1] >= Ui - P[0];
        const bool f1 = P[3] >= Ui - P[2];
        int off = f1 ? 1 : 2;
        off = f0 ? 0 : off;
        if (off == 2) {
            const bool f2 = P[5] >= Ui - P[4];
            const bool f3 = P[7] >= Ui - P[6];
            off = f3 ? 3 : 4;
            off = f2 ? 2 : off;
        }
        int c = a + off;
        if (off == 4) {
            // rare: crossing in (a+3, i]; i passes without a look
            int lo = c, b = i, step = 1;
            while (lo < b) {
                int p = lo + step - 1;
                p = p < b - 1 ? p : b - 1;
                if (UD[2 * p + 1] >= Ui - UD[2 * p]) { b = p; break; }
                lo = p + 1;
                step <<= 1;
            }
            while (lo < b) {
                const int mid = (lo + b) >> 1;
                if (UD[2 * mid + 1] >= Ui - UD[2 * mid]) b = mid; else lo = mid + 1;
            }
            c = lo;
        }
        jp = c;
        const double dc = UD[2 * c + 1];
        const double t = Ui - UD[2 * c - 2];
        v = (c >= k && t < dc) ? t : dc;
    }
    // every lane has read row k-1 (gallop included) before any lane
    // overwrites it: the store stays after the branch
    __asm__ volatile("" ::: "memory");
    if (act) UD[2 * i + 1] = v;
}

// Bottleneck W*(pp) = D_pp(L) for the degrees in `tm`, handed to
// on_target(pp, W, tm) as soon as row pp is done; it returns the degrees
// still wanted (it may drop larger ones), and rows stop after the last.  Row
// k is evaluated for i in [k, L - tau(k) + k] only, tau(k) the smallest wanted
// degree >= k: larger i cannot reach a wanted cell.  Lane l of row k takes
// i = k + l (+64): the window width never grows with k, so after the first
// rows one pass covers a row, and a lane's crossing from row k-1 (for i-1) is
// a lower bound for row k.  After each row, D[hi+1] = +inf marks the first
// position the row did not reach.
template <class OnTarget>
__device__ void solve_dp(WaveLds& Wv, int L, Mask tm, int lane, OnTarget&& on_target)
{
    double* UD = Wv.UD;
    int tau = tm.next(1);
    if (tau == 0) return;
    unsigned n_ent = 0;
    {
        const int hi = L - tau + 1;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int i = 1 + lane + 64 * s;
            if (i <= hi) UD[2 * i + 1] = UD[2 * i];
        }
        if (lane == 0) UD[2 * hi + 3] = kInf;
        n_ent += (unsigned)hi;
        wave_sync();
        if (tau == 1) {
            tm = on_target(1, UD[2 * L], tm);
            tau = tm.next(2);
        }
    }
    int jp0 = 0, jp1 = 0;
    for (int k = 2; tau != 0; ++k) {
        const int hi = L - tau + k;
        // lower bounds: own crossing (i-1, row k-1) and the next lane's (i, row k-1)
        const int top1 = __builtin_amdgcn_readlane(jp1, 0);
        const int nb0 = from_next_lane(jp0, top1);
        const int lb0 = jp0 > nb0 ? jp0 : nb0;
        if (hi - k >= 64) {                    // high part first: in place
            const int nb1 = from_next_lane(jp1, jp1);
            dp_entry(UD, k, hi, k + 64 + lane, jp1 > nb1 ? jp1 : nb1, jp1);
        }
        dp_entry(UD, k, hi, k + lane, lb0, jp0);
        if (lane == 0) UD[2 * hi + 3] = kInf;
        n_ent += (unsigned)(hi - k + 1);
        wave_sync();
        if (k == tau) {
            tm = on_target(k, UD[2 * L + 1], tm);
            tau = tm.next(k + 1);
        }
    }
    tally(Wv, lane, kDpEntries, n_ent);
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

// The successor tables of threshold W: level s of J holds next^(2^s), next(e)
// the smallest c with U_e - U_c <= W (node 0 maps to itself), for levels
// 0 .. levels-1.
template <int S>
__device__ void successor_tables(const double* U, uint8_t* J, int lane, int L, int levels, double W)
{
    // next(e): the failing c (U_e - U_c > W) form a prefix of [0, e); c = e-1
    // passes when W is at least every single-layer cost, and so does every
    // c > e-1 (U is non-decreasing and +inf past L)
    // binary lifting of both halves in step (lanes past L read the +inf
    // padding and store nothing)
    const bool two = L > 64;
    const int e0 = 1 + lane, e1 = 65 + lane;
    int cur0 = 0, cur1 = 0;
    {
        const double Ue0 = U[e0 * S];
        if (two) {
            const double Ue1 = U[e1 * S];
            cur1 = Ue1 - U[63 * S] > W ? 64 : 0;
#pragma unroll
            for (int step = 32; step >= 1; step >>= 1) {
                const bool g0 = Ue0 - U[(cur0 + step - 1) * S] > W;
                const bool g1 = Ue1 - U[(cur1 + step - 1) * S] > W;
                cur0 += g0 ? step : 0;
                cur1 += g1 ? step : 0;
            }
        } else {
#pragma unroll
            for (int step = 32; step >= 1; step >>= 1)
                cur0 += Ue0 - U[(cur0 + step - 1) * S] > W ? step : 0;
        }
    }
    // lanes past L follow node 0 (a fixed point) so every read stays in range
    cur0 = e0 <= L ? cur0 : 0;
    cur1 = (two && e1 <= L) ? cur1 : 0;
    if (e0 <= L) J[e0] = (uint8_t)cur0;
    if (two && e1 <= L) J[e1] = (uint8_t)cur1;
    if (lane < levels) J[lane * kLevelStride] = 0;
    wave_sync();
    for (int s = 1; s < levels; ++s) {
        const uint8_t* prev = J + (s - 1) * kLevelStride;
        uint8_t* lev = J + s * kLevelStride;
        cur0 = prev[cur0];
        if (two) cur1 = prev[cur1];
        if (e0 <= L) lev[e0] = (uint8_t)cur0;
        if (two && e1 <= L) lev[e1] = (uint8_t)cur1;
        wave_sync();
    }
}

// The cuts of the canonical split of pp >= 2 stages from successor tables of
// levels 32 - clz(pp - 1): c_k for k = lane (cA) and k = lane + 64 (cB);
// c_0 = 0, c_pp = L, and 0 for k > pp.  Every lane walks (nodes stay in
// [0, L]); only lanes 1 <= k < pp keep the result.
__device__ __forceinline__ void cuts_from_tables(const uint8_t* J, int lane, int L, int pp, int levels, int& cA_out,
                                                 int& cB_out)
{
    const bool hi_half = pp >= 64;
    const int k0 = lane, k1 = lane + 64;
    const int d0 = pp - k0, d1 = pp - k1;
    int n0 = L, n1 = L;
    for (int s = 0; s < levels; ++s) {
        const uint8_t* lev = J + s * kLevelStride;
        const int nd0 = lev[n0];
        n0 = ((d0 >> s) & 1) ? nd0 : n0;
        if (hi_half) {
            const int nd1 = lev[n1];
            n1 = ((d1 >> s) & 1) ? nd1 : n1;
        }
    }
    int cA = (k0 >= 1 && k0 < pp) ? (n0 > k0 ? n0 : k0) : 0;
    cA = k0 == pp ? L : cA;
    int cB = 0;
    if (hi_half) {
        cB = k1 < pp ? (n1 > k1 ? n1 : k1) : 0;
        cB = k1 == pp ? L : cB;
    }
    cA_out = cA;
    cB_out = cB;
}

// The stages of the split with cuts cA (c_k, k = lane) and cB (k = lane + 64):
// stage s ends where stage s+1 starts, at the next lane's cut (lane 63 of the
// low half takes c_64, lane 63 of the high half c_128).
__device__ __forceinline__ Stages stages_from_cuts(int cA, int cB, int L, int pp)
{
    Stages r;
    r.lo0 = cA;
    r.hi0 = from_next_lane(cA, __builtin_amdgcn_readlane(cB, 0));
    r.lo1 = cB;
    r.hi1 = from_next_lane(cB, pp == 128 ? L : 0);
    return r;
}

__device__ __forceinline__ Stages stages_from_tables(const uint8_t* J, int lane, int L, int pp, int levels)
{
    int cA, cB;
    cuts_from_tables(J, lane, L, pp, levels, cA, cB);
    return stages_from_cuts(cA, cB, L, pp);
}

template <int S>
__device__ Stages canonical_stages(const double* U, uint8_t* J, int lane, int L, int pp, double W)
{
    if (pp == 1) {
        Stages r;
        r.lo0 = 0; r.hi0 = L; r.lo1 = 0; r.hi1 = 0;
        return r;
    }
    const int levels = 32 - __clz(pp - 1);   // 2^levels > pp - 1
    successor_tables<S>(U, J, lane, L, levels, W);
    return stages_from_tables(J, lane, L, pp, levels);
}

constexpr int kPureCachedDegrees = 96;

// The pure-compute problem's canonical split of pp >= 2 stages (the cuts of
// its prefix Upure at its bottleneck wpure = Wpure(pp)).  It depends on
// neither the count, nor the contention, nor the tensor degree, so the block
// keeps it, once computed for its current item, in its rows of a global cache
// (row pp: the bytes c_0 .. c_pp), and bit pp - 1 of `cached` (LDS, cleared
// per item) says that the row is current.  Two waves that miss together both
// write the same bytes.  Degrees above kPureCachedDegrees are recomputed: few
// items use them, so their rows leave L2 between uses and each write of one
// came back as HBM write-back (a fifth of the kernel's traffic) while saving
// little time.
__device__ Stages pure_split(const double* Upure, double wpure, unsigned long long* cached, WaveLds& Wv,
                             uint8_t* cache, int lane, int L, int pp)
{
    static_assert(kLmax * (kLmax + 1) / 2 - 3 + kLmax + 1 <= kPureCutBytes, "cache rows");
    uint8_t* row = cache + (pp * (pp + 1) / 2 - 3);
    unsigned long long* word = &cached[(pp - 1) >> 6];
    const unsigned long long bit = 1ull << ((pp - 1) & 63);
    const unsigned long long w = __hip_atomic_load(word, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
    const bool hit = pp <= kPureCachedDegrees && __builtin_amdgcn_readfirstlane((int)((w & bit) != 0ull)) != 0;
    int cA, cB;
    if (hit) {
        cA = lane <= pp ? (int)row[lane] : 0;
        cB = lane + 64 <= pp ? (int)row[lane + 64] : 0;
    } else {
        const int levels = 32 - __clz(pp - 1);   // 2^levels > pp - 1
        successor_tables<1>(Upure, Wv.J, lane, L, levels, wpure);
        cuts_from_tables(Wv.J, lane, L, pp, levels, cA, cB);
        if (pp <= kPureCachedDegrees) {
            if (lane <= pp) row[lane] = (uint8_t)cA;
            if (lane + 64 <= pp) row[lane + 64] = (uint8_t)cB;
            // the row's stores before the bit
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            if (lane == 0) __hip_atomic_fetch_or(word, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
    }
    return stages_from_cuts(cA, cB, L, pp);
}

// Does every split of the L layers into pp stages have a stage costing more
// than th (a stage's cost a difference of U, stride S, as the recursion forms
// it)?  Right to left, prev(e) is the smallest c with U_e - U_c <= th (e
// itself when layer e-1 alone exceeds th): the fewest stages with costs <= th
// take prev steps from L to 0, and a split into fewer stages refines into pp
// (costs only fall), so the answer is no exactly when prev^(pp-1)(L) reaches
// a node n with prev(n) = 0.  prev^(2^s) tables by binary lifting as in
// canonical_stages, one walk.  Uniform result.
template <int S>
__device__ bool bottleneck_exceeds(const double* U, uint8_t* J, int lane, int L, int pp, double th)
{
    if (th < 0.0) return true;         // every stage costs at least 0
    if (!(th >= 0.0)) return false;
    // from here c = e passes for every e, so prev(e) <= e <= L: every node
    // and table entry stays in [0, L]
    const int levels = pp > 1 ? 32 - __clz(pp - 1) : 1;   // 2^levels > pp - 1
    successor_tables<S>(U, J, lane, L, levels, th);
    int n = L;
    for (int s = 0; s < levels; ++s)
        if (((pp - 1) >> s) & 1) n = J[s * kLevelStride + n];
    const bool ok = n == 0 || J[n] == 0;
    wave_sync();
    return !ok;
}

// The largest stage cost, on the problem's prefix U (stride 2), of split sg.
__device__ __forceinline__ double split_cost(const double* UD, const Stages& sg, int lane, int pp)
{
    double c = 0.0;
    if (lane < pp) c = UD[2 * sg.hi0] - UD[2 * sg.lo0];
    if (lane + 64 < pp) c = fmax(c, UD[2 * sg.hi1] - UD[2 * sg.lo1]);
    const double ub = wave_reduce1<OpMax>(c);
    wave_sync();
    return ub;
}

// The bottleneck of pp stages over the problem's prefix U (stride 2) when a
// few splits certify it, else -1.  The first is sgp, the pure-compute
// problem's canonical split (cuts of its prefix at its bottleneck Wpure(pp)):
// it costs UB on U, so the bottleneck is at most UB; if no split keeps every
// stage below UB (the test above at the largest double under UB) the
// bottleneck is UB exactly.  Otherwise some split does, and the canonical
// split of U under that double costs less than UB: it is the next one tried.
// Returns -2 when no microbatch count can fit the degree's plans: a canonical
// split at a threshold of at least the bottleneck has its cuts at or left of
// the bottleneck's, so its first stage is contained in the priced split's first
// stage; if that smaller stage already overflows memory with the largest
// admissible count (minf = min(m, pp) microbatches in flight, bm samples each,
// cap = mem tp, the pricing's test term by term), so does the priced one, and
// with every smaller count too (MEMTEST: the test is made).
template <int ROUNDS = kCertRounds, bool MEMTEST = false>
__device__ double certified_bottleneck(Stages sgp, WaveLds& Wv, int lane, int L, int pp, const double* Pp = nullptr,
                                       const double* Ap = nullptr, double cap = kInf, double bm = 0.0, int minf = 0)
{
    double ub = split_cost(Wv.UD, sgp, lane, pp);
    for (int r = 0;; ++r) {
        if (!(ub > 0.0 && ub < kInf)) return -1.0;
        const double below = __longlong_as_double(__double_as_longlong(ub) - 1);
        if (bottleneck_exceeds<2>(Wv.UD, Wv.J, lane, L, pp, below)) return ub;
        // a split with every stage at most `below` exists, and every single
        // layer costs at most that (else the test would have passed): the
        // test's tables are those of its canonical split
        if (!MEMTEST && r + 1 == ROUNDS) return -1.0;
        const Stages sg = stages_from_tables(Wv.J, lane, L, pp, 32 - __clz(pp - 1));
        if constexpr (MEMTEST) {
            const int c1 = __builtin_amdgcn_readfirstlane(sg.hi0);   // lane 0: stage 0 = [0, c_1)
            const double i0 = (double)minf * bm;
            if (4.0 * Pp[c1] + i0 * Ap[c1] > cap) return -2.0;
            if (r + 1 == ROUNDS) return -1.0;
        }
        ub = split_cost(Wv.UD, sg, lane, pp);
    }
}

// ------------------------------------------------------------ memory-constrained partition

// Stage [j, e) fits when 4 P + ib A <= cap, ib = in-flight microbatches x
// samples per microbatch and cap = mem x tp (the memory check of the pricing,
// same operation order).
__device__ __forceinline__ bool seg_fits(double Pe, double Ae, double Pj, double Aj, double ib, double cap)
{
    return 4.0 * (Pe - Pj) + ib * (Ae - Aj) <= cap;
}

// Stage bounds of a cut vector held as c_k in lane k (cA) and lane k - 64
// (cB), c_0 = 0 and c_pp = L set here; as canonical_stages returns them.
__device__ __forceinline__ Stages stages_from_cuts(int cA, int cB, int lane, int L, int pp)
{
    cA = (lane >= 1 && lane < pp) ? cA : 0;
    cA = lane == pp ? L : cA;
    cB = lane + 64 < pp ? cB : 0;
    cB = lane + 64 == pp ? L : cB;
    Stages r;
    r.lo0 = cA;
    r.hi0 = from_next_lane(cA, __builtin_amdgcn_readlane(cB, 0));
    r.lo1 = cB;
    r.hi1 = from_next_lane(cB, pp == 128 ? L : 0);
    return r;
}

// Do the stages of sg all fit with m microbatches of b samples?  Stage s
// holds min(m, pp - s) microbatches.
__device__ __forceinline__ bool stages_fit(const Stages& sg, const double* Pp, const double* Ap, int lane,
                                           int pp, int m, double b, double cap)
{
    bool bad = false;
    if (lane < pp) {
        const int r = pp - lane;
        bad = !seg_fits(Pp[sg.hi0], Ap[sg.hi0], Pp[sg.lo0], Ap[sg.lo0], (double)(m < r ? m : r) * b, cap);
    }
    if (lane + 64 < pp) {
        const int r = pp - lane - 64;
        bad |= !seg_fits(Pp[sg.hi1], Ap[sg.hi1], Pp[sg.lo1], Ap[sg.lo1], (double)(m < r ? m : r) * b, cap);
    }
    return __ballot(bad) == 0ull;
}

// Lexicographically smallest cut vector of pp stages whose every stage fits
// (stage k holds min(m, pp - k) microbatches of b samples) and costs at most
// W, if there is one (W = +inf: memory alone).  From the back, the t-th stage
// starts at r_t, the leftmost start whose stage up to r_{t-1} fits and costs
// at most W (both hold on a suffix of starts: cost and memory only grow as a
// stage extends left); then c_k = max(k, r_{pp-k}).  If any split fits
// within W, no cut of it lies left of this vector's, and this vector fits
// too: a stage the clamp leaves as one layer holds no more microbatches than
// the stage holding that layer in the other split.  So the split exists iff
// the vector passes the final check.  Lane l tests starts l and l + 64.
template <int S>
__device__ bool mem_cuts(const double* U, const double* Pp, const double* Ap, int lane, int L, int pp, int m,
                         double b, double cap, double W, Stages& sg)
{
    const int j0 = lane, j1 = lane + 64;
    const double Uj0 = U[j0 * S], Uj1 = U[j1 * S];
    const double Pj0 = Pp[j0], Aj0 = Ap[j0];
    const double Pj1 = j1 <= kLmax ? Pp[j1] : 0.0, Aj1 = j1 <= kLmax ? Ap[j1] : 0.0;
    int cA = 0, cB = 0;
    int e = L;
    for (int t = 1; t < pp; ++t) {
        int r = 0;
        if (e > 0) {
            const double ib = (double)(m < t ? m : t) * b;
            const double Ue = U[e * S], Pe = Pp[e], Ae = Ap[e];
            const bool p0 = j0 < e && Ue - Uj0 <= W && seg_fits(Pe, Ae, Pj0, Aj0, ib, cap);
            const bool p1 = j1 < e && Ue - Uj1 <= W && seg_fits(Pe, Ae, Pj1, Aj1, ib, cap);
            const unsigned long long b0 = __ballot(p0), b1 = __ballot(p1);
            if (b0) r = __ffsll((long long)b0) - 1;
            else if (b1) r = 63 + __ffsll((long long)b1);
            else return false;        // not even the last layer alone: no split
        }
        const int k = pp - t;
        const int c = r > k ? r : k;
        cA = lane == k ? c : cA;
        cB = lane + 64 == k ? c : cB;
        e = r;
    }
    sg = stages_from_cuts(cA, cB, lane, L, pp);
    bool bad = false;
    if (lane < pp) {
        const int r = pp - lane;
        bad = !(sg.hi0 > sg.lo0) || !(U[sg.hi0 * S] - U[sg.lo0 * S] <= W) ||
              !seg_fits(Pp[sg.hi0], Ap[sg.hi0], Pp[sg.lo0], Ap[sg.lo0], (double)(m < r ? m : r) * b, cap);
    }
    if (lane + 64 < pp) {
        const int r = pp - lane - 64;
        bad |= !(sg.hi1 > sg.lo1) || !(U[sg.hi1 * S] - U[sg.lo1 * S] <= W) ||
               !seg_fits(Pp[sg.hi1], Ap[sg.hi1], Pp[sg.lo1], Ap[sg.lo1], (double)(m < r ? m : r) * b, cap);
    }
    return __ballot(bad) == 0ull;
}

// Smallest starting position j in [0, i] of a stage ending at i that fits
// with ib (j = i, the empty stage, always does).
__device__ __forceinline__ int fit_start(const double* Pp, const double* Ap, int i, double Pi, double Ai,
                                         double ib, double cap)
{
    int lo = 0, hi = i;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (seg_fits(Pi, Ai, Pp[mid], Ap[mid], ib, cap)) hi = mid; else lo = mid + 1;
    }
    return lo;
}

// One entry of row k of the memory-constrained recursion (R holds row k-1
// and receives row k in place, as in dp_entry):
//   D_k(i) = min over j in [a, i-1] of max(D_{k-1}(j), U_i - U_j),
// a = max(k-1, the first start whose stage up to i fits as stage k-1).
// D_{k-1} is non-decreasing in j also under the memory limits (dropping the
// last layer of a prefix, or splitting a stage to keep k-1 of them, moves
// stages only towards the back, where they hold fewer microbatches), so the
// minimum sits at the crossing c, the first j >= a with D_{k-1}(j) >=
// U_i - U_j (i itself counts as passing): min(D_{k-1}(c), U_i - U_{c-1}),
// each term only where its position lies in the window.
template <int S>
__device__ __forceinline__ void mem_entry(const double* U, double* R, int k, int hk, int i, double Ui, int fs)
{
    double v = kInf;
    const bool act = i <= hk;
    if (act) {
        const int a = fs > k - 1 ? fs : k - 1;
        if (i >= k && a < i) {
            int lo = a, hi = i;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (R[mid] >= Ui - U[mid * S]) hi = mid; else lo = mid + 1;
            }
            v = lo < i ? R[lo] : kInf;
            if (lo > a) v = fmin(v, Ui - U[(lo - 1) * S]);
        }
    }
    __asm__ volatile("" ::: "memory");
    if (act) R[i] = v;
}

// Bottleneck of pp stages over the splits whose every stage fits (stage k
// holds min(m, pp - k) microbatches of b samples): D_pp(L), +inf if none.
// R: the wave's row of kLmax + 1 doubles.  Lane l owns i = 1 + l and 65 + l.
// Row k is needed only up to i = L - (pp - k) (each later stage takes a
// layer), which is also as far as row k + 1 reads it.
template <int S>
__device__ double mem_bottleneck(const double* U, const double* Pp, const double* Ap, double* R, int lane,
                                 int L, int pp, int m, double b, double cap, unsigned& entries)
{
    const int i0 = 1 + lane, i1 = 65 + lane;
    const double Ui0 = U[i0 * S], Ui1 = U[i1 * S];
    const double Pi0 = Pp[i0], Ai0 = Ap[i0];
    const double Pi1 = i1 <= kLmax ? Pp[i1] : 0.0, Ai1 = i1 <= kLmax ? Ap[i1] : 0.0;
    const bool two = L > 64;
    // row 1: the first stage holds min(m, pp) microbatches
    int rcur = m < pp ? m : pp;
    double ib = (double)rcur * b;
    int fs0 = i0 <= L ? fit_start(Pp, Ap, i0, Pi0, Ai0, ib, cap) : 0;
    int fs1 = (two && i1 <= L) ? fit_start(Pp, Ap, i1, Pi1, Ai1, ib, cap) : 0;
    const int h1 = L - pp + 1;
    if (lane == 0) R[0] = kInf;
    if (i0 <= h1) R[i0] = fs0 == 0 ? Ui0 - U[0] : kInf;
    if (two && i1 <= h1) R[i1] = fs1 == 0 ? Ui1 - U[0] : kInf;
    unsigned n = (unsigned)h1;
    wave_sync();
    for (int k = 2; k <= pp; ++k) {
        const int r = m < pp - k + 1 ? m : pp - k + 1;
        if (r != rcur) {
            rcur = r;
            ib = (double)r * b;
            fs0 = i0 <= L ? fit_start(Pp, Ap, i0, Pi0, Ai0, ib, cap) : 0;
            fs1 = (two && i1 <= L) ? fit_start(Pp, Ap, i1, Pi1, Ai1, ib, cap) : 0;
        }
        const int hk = L - pp + k;
        if (hk >= 65) mem_entry<S>(U, R, k, hk, i1, Ui1, fs1);   // high half first: reads only lower positions
        mem_entry<S>(U, R, k, hk, i0, Ui0, fs0);
        n += (unsigned)(hk - k + 1);
        wave_sync();
    }
    entries += n;
    const double W = R[L];
    wave_sync();
    return W;
}

// Per-sample p2p bytes and largest stage parameters of the stages in sg
// (as the pricing sums them).
__device__ __forceinline__ void stage_sums(const Stages& sg, const float* x, const double* Pp, int lane, int pp,
                                           double& sumX, double& pmax)
{
    double P0 = 0.0, P1 = 0.0, sx = 0.0;
    if (lane < pp) {
        P0 = Pp[sg.hi0] - Pp[sg.lo0];
        if (lane < pp - 1) sx = (double)x[sg.hi0 - 1];
    }
    if (lane + 64 < pp) {
        P1 = Pp[sg.hi1] - Pp[sg.lo1];
        if (lane + 64 < pp - 1) sx += (double)x[sg.hi1 - 1];
    }
    double rs[1] = {sx}, rm[1] = {fmax(P0, P1)};
    wave_reduce<OpSum, 1>(rs);
    wave_reduce<OpMax, 1>(rm);
    sumX = rs[0];
    pmax = rm[0];
}

// The memory rule's counts of one degree: ranks lo-1 down to 0 of the
// wave's admissible list (bq, mq), whose balanced split does not fit.  Each
// is skipped when a lower bound of its time with any split (as target_bound,
// with the unconstrained bottleneck W) lies past lim_c; otherwise its
// fitting splits are tested (none: no smaller count fits either, stop), its
// bottleneck solved and its lexicographically smallest cuts priced into plan
// slot base + rank.  Out of line so that its registers do not add to those
// live around the pricing.  Returns the least of best_t and the times priced.
template <class T>
using Lds = __attribute__((address_space(3))) T;

template <int S>
__device__ __noinline__ double mem_counts(const Lds<double>* Ul, const Lds<double>* Ppl, const Lds<double>* Apl,
                                          const Lds<float>* xl, Lds<double>* Rl, Lds<WaveLds>* Wpl, int lane, int L,
                                          int tp, int pp, int dp, int lo, int base, double W, double cap,
                                          double sumS, double c_p2p, double c_ar, double plb, double x_min,
                                          double best_t, double lim_c, double tie_eps, bool prune, bool keep_cuts)
{
    // the pointers arrive typed as LDS so that the accesses below stay LDS
    // accesses in this out-of-line function
    const double* U = (const double*)Ul;
    const double* Pp = (const double*)Ppl;
    const double* Ap = (const double*)Apl;
    const float* x = (const float*)xl;
    double* R = (double*)Rl;
    WaveLds& Wv = *(WaveLds*)Wpl;
    const double fill_lb = sumS + c_p2p * ((double)(pp - 1) * x_min);
    for (int rk = lo - 1; rk >= 0; --rk) {
        const double bm = Wv.bq[rk];
        const int m = Wv.mq[rk];
        if (lim_c < kInf && (bm * fill_lb + (double)(m - 1) * (bm * W) + plb * c_ar) * (1.0 - 1e-9) > lim_c)
            continue;
        Stages sm;
        tally(Wv, lane, kAlgOps, 4ull * (unsigned)L);
        if (!mem_cuts<S>(U, Pp, Ap, lane, L, pp, m, bm, cap, kInf, sm)) break;
        unsigned ent = 0;
        const double Wm = mem_bottleneck<S>(U, Pp, Ap, R, lane, L, pp, m, bm, cap, ent);
        tally(Wv, lane, kDpEntries, ent);
        tally(Wv, lane, kMemParts, 1);
        tally(Wv, lane, kAlgOps, 4ull * (unsigned)L);
        if (!(Wm < kInf) || !mem_cuts<S>(U, Pp, Ap, lane, L, pp, m, bm, cap, Wm, sm)) continue;
        double sX, pm;
        stage_sums(sm, x, Pp, lane, pp, sX, pm);
        const double Tm = bm * (sumS + c_p2p * sX) + (double)(m - 1) * (bm * Wm) + ((dp > 1) ? pm * c_ar : 0.0);
        if (lane == 0 && base + rk < kMaxPlans) Wv.planT[base + rk] = Tm;
        best_t = fmin(best_t, Tm);
        if (prune) lim_c = fmin(lim_c, Tm * (1.0 + tie_eps));
        if (keep_cuts && Tm < Wv.cut_T) {
            if (lane < pp - 1) Wv.cutrow[lane] = (uint8_t)sm.hi0;
            if (lane + 64 < pp - 1) Wv.cutrow[lane + 64] = (uint8_t)sm.hi1;
            if (lane == 0) {
                Wv.cut_T = Tm;
                Wv.cut_tp = tp;
                Wv.cut_pp = pp;
                Wv.cut_m = m;
            }
        }
        wave_sync();
    }
    return best_t;
}

// ------------------------------------------------------------ exact-T partition

// The exact-T rule: the split minimising the plan's whole iteration time
// among the splits whose every stage fits memory.  The stage costs summed over
// the stages do not depend on the split (the stages tile the layers), so the
// split minimises Phi = (cS Smax + cX X) + cP Pmax: Smax the slowest stage
// per sample, X the boundary bytes x_{c_1-1} + (x_{c_2-1} + ...) added from
// the back, Pmax the largest stage's parameter bytes, with the coefficients
// of the steady state, the fill's point-to-point and the all-reduce (Sec. 3.4,
// Eq. 4).  Ties: the least (Phi, Smax, Pmax, X), then the lexicographically
// smallest cuts.  A stage's parameter and activation bytes are differences of
// the running totals Pp, Ap; memory as the pricing: 4 P / tp + min(m, pp-k)
// b A / tp <= mem for stage k.
struct ExtCtx {
    int L, pp, m;
    double b, tpd, mem;
    double cS, cX, cP;
};

struct ExtKey {
    double phi, s, p, x;
};

__device__ __forceinline__ bool ext_less(const ExtKey& a, const ExtKey& b)
{
    if (a.phi != b.phi) return a.phi < b.phi;
    if (a.s != b.s) return a.s < b.s;
    if (a.p != b.p) return a.p < b.p;
    return a.x < b.x;
}

__device__ __forceinline__ double ext_phi(const ExtCtx& E, double sm, double x, double pm)
{
    return (E.cS * sm + E.cX * x) + E.cP * pm;
}

// Stage [i, e) as stage k within the thresholds: cost at most tS, parameter
// bytes at most tP, and it fits memory (each holds on a prefix of the ends e).
template <int S>
__device__ __forceinline__ bool ext_ok(const ExtCtx& E, const double* U, const double* Pp, const double* Ap, int i,
                                       int e, int k, double tS, double tP)
{
    const double P = Pp[e] - Pp[i];
    const double Am = Ap[e] - Ap[i];
    const int r = E.pp - k;
    const int infl = E.m < r ? E.m : r;
    const double mem = 4.0 * P / E.tpd + (double)infl * E.b * Am / E.tpd;
    return U[e * S] - U[i * S] <= tS && P <= tP && mem <= E.mem;
}

// Suffix recursion over the splits within the thresholds, rows t = 1..tmax
// into H (L + 1 doubles, in place: row t at i reads row t-1 only right of i):
//   KIND 0: H_t(i) = least X of layers [i, L) as the last t stages,
//           H_1(i) = 0, H_t(i) = min_e x_{e-1} + H_{t-1}(e);
//   KIND 1: H_t(i) = least largest stage parameter bytes of that suffix,
//           H_1(i) = P(i, L), H_t(i) = min_e max(P(i, e), H_{t-1}(e));
//   KIND 2: the same with the stages' per-sample costs;
// over the ends e whose stage [i, e) is allowed as stage pp - t (+inf: none).
// Returns H_tmax(0).  Lanes own i = lane and lane + 64 and scan their ends in
// step, stopping at the first stage not allowed.
template <int S, int KIND>
__device__ double ext_rows(const ExtCtx& E, const double* U, const double* Pp, const double* Ap, const float* x,
                           double* H, int lane, double tS, double tP, int tmax)
{
    const int L = E.L, pp = E.pp;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int i = lane + 64 * h;
        if (i <= L) {
            double v = kInf;
            if (i < L && ext_ok<S>(E, U, Pp, Ap, i, L, pp - 1, tS, tP))
                v = KIND == 0 ? 0.0 : (KIND == 1 ? Pp[L] - Pp[i] : U[L * S] - U[i * S]);
            H[i] = v;
        }
    }
    wave_sync();
    for (int t = 2; t <= tmax; ++t) {
        const int k = pp - t, last = L - t + 1;
        const int i0 = lane, i1 = lane + 64;
        double b0 = kInf, b1 = kInf;
        bool g0 = i0 <= L - t, g1 = i1 <= L - t;
        int e0 = i0 + 1, e1 = i1 + 1;
        while (g0 || g1) {
            if (g0) {
                if (e0 > last || !ext_ok<S>(E, U, Pp, Ap, i0, e0, k, tS, tP)) {
                    g0 = false;
                } else {
                    const double h = H[e0];
                    if (h < kInf)
                        b0 = fmin(b0, KIND == 0 ? (double)x[e0 - 1] + h
                                                : fmax(KIND == 1 ? Pp[e0] - Pp[i0] : U[e0 * S] - U[i0 * S], h));
                    ++e0;
                }
            }
            if (g1) {
                if (e1 > last || !ext_ok<S>(E, U, Pp, Ap, i1, e1, k, tS, tP)) {
                    g1 = false;
                } else {
                    const double h = H[e1];
                    if (h < kInf)
                        b1 = fmin(b1, KIND == 0 ? (double)x[e1 - 1] + h
                                                : fmax(KIND == 1 ? Pp[e1] - Pp[i1] : U[e1 * S] - U[i1 * S], h));
                    ++e1;
                }
            }
        }
        // every lane has read row t-1 before any lane overwrites it
        __asm__ volatile("" ::: "memory");
        if (i0 <= L) H[i0] = i0 <= L - t ? b0 : kInf;
        if (i1 <= L) H[i1] = i1 <= L - t ? b1 : kInf;
        wave_sync();
    }
    const double r = H[0];
    wave_sync();
    return r;
}

// The least value V(s, e) = V[e] - V[s] (element e at V[e * VS]) of any
// segment above th (+inf if none): each lane bisects the ends of its starts.
template <int VS>
__device__ double ext_next(const double* V, int lane, int L, double th)
{
    double best = kInf;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int s = lane + 64 * h;
        if (s < L) {
            const double Vs = V[s * VS];
            int lo = s + 1, hi = L + 1;          // first e in [s+1, L] with V(s, e) > th, L + 1: none
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (V[mid * VS] - Vs > th) hi = mid; else lo = mid + 1;
            }
            if (lo <= L) best = fmin(best, V[lo * VS] - Vs);
        }
    }
    return wave_reduce1<OpMin>(best);
}

// Exact-T key of one plan (false: no split fits).  Thresholds are visited by
// tS then tP ascending; each pair's least X gives the key ((cS tS + cX X) +
// cP tP, tS, tP, X), and the least key over the pairs is the least key over
// the splits.  A pair after the best key found so far wins only with a
// smaller Phi, so the visit stops where a lower bound of Phi reaches the best:
//   tS runs from the least Smax of any split that fits and stops once (cS tS
//   + cX Xlo) + cP Plo reaches the best (Xlo, Plo the least X and Pmax of any
//   split that fits), or, when cS = 0, once the best is the least Phi of any
//   split;
//   tP runs from the least Pmax within tS and stops once (cS tS + cX Xs) +
//   cP tP reaches the best (Xs the least X within tS) or its X is Xs.
template <int S>
__device__ bool ext_solve(const ExtCtx& E, const double* U, const double* Pp, const double* Ap, const float* x,
                          double* H, int lane, ExtKey& best)
{
    const double p_lo = ext_rows<S, 1>(E, U, Pp, Ap, x, H, lane, kInf, kInf, E.pp);
    if (!(p_lo < kInf)) return false;
    const double s_lo = ext_rows<S, 2>(E, U, Pp, Ap, x, H, lane, kInf, kInf, E.pp);
    const double x_lo = ext_rows<S, 0>(E, U, Pp, Ap, x, H, lane, kInf, kInf, E.pp);
    double phi_all = kInf;
    if (E.cS == 0.0) {
        for (double tP = p_lo; tP < kInf; tP = ext_next<1>(Pp, lane, E.L, tP)) {
            const double X = ext_rows<S, 0>(E, U, Pp, Ap, x, H, lane, kInf, tP, E.pp);
            if (X < kInf) phi_all = fmin(phi_all, (0.0 + E.cX * X) + E.cP * tP);
            if (X == x_lo) break;
        }
    }
    bool found = false;
    for (double tS = s_lo; tS < kInf; tS = ext_next<S>(U, lane, E.L, tS)) {
        if (found && (E.cS == 0.0 ? best.phi <= phi_all : ext_phi(E, tS, x_lo, p_lo) >= best.phi)) break;
        const double pmin = ext_rows<S, 1>(E, U, Pp, Ap, x, H, lane, tS, kInf, E.pp);
        if (!(pmin < kInf)) continue;
        const double xs = ext_rows<S, 0>(E, U, Pp, Ap, x, H, lane, tS, kInf, E.pp);
        for (double tP = pmin; tP < kInf; tP = ext_next<1>(Pp, lane, E.L, tP)) {
            if (found && ext_phi(E, tS, xs, tP) >= best.phi) break;
            const double X = ext_rows<S, 0>(E, U, Pp, Ap, x, H, lane, tS, tP, E.pp);
            if (X < kInf) {
                const ExtKey k = {ext_phi(E, tS, X, tP), tS, tP, X};
                if (!found || ext_less(k, best)) {
                    best = k;
                    found = true;
                }
            }
            if (X == xs) break;
        }
    }
    return found;
}

// The lexicographically smallest split of least X within the key's
// thresholds, cut by cut from the left: c_k is the first end e of an allowed
// stage k-1 from c_{k-1} with x_{e-1} + H_{pp-k}(e) equal to the X left.
// The suffix rows are recomputed for each cut.  Returns the stage bounds.
template <int S>
__device__ Stages ext_cuts(const ExtCtx& E, const double* U, const double* Pp, const double* Ap, const float* x,
                           double* H, int lane, const ExtKey& key)
{
    int cA = 0, cB = 0;
    int i = 0;
    double rest = key.x;
    for (int k = 1; k < E.pp; ++k) {
        const int t = E.pp - k + 1;
        ext_rows<S, 0>(E, U, Pp, Ap, x, H, lane, key.s, key.p, t - 1);
        int c = -1;
        for (int base = i + 1; base <= E.L - t + 1 && c < 0; base += 64) {
            const int e = base + lane;
            bool ok = false;
            if (e <= E.L - t + 1 && ext_ok<S>(E, U, Pp, Ap, i, e, k - 1, key.s, key.p)) {
                const double h = H[e];
                ok = h < kInf && (double)x[e - 1] + h == rest;
            }
            const unsigned long long bm = __ballot(ok);
            if (bm) c = base + __ffsll((long long)bm) - 1;
        }
        // a split of the key exists, so some end passes; keep the cuts ordered regardless
        c = c < 0 ? i + 1 : c;
        rest = H[c];
        wave_sync();
        cA = lane == k ? c : cA;
        cB = lane + 64 == k ? c : cB;
        i = c;
    }
    return stages_from_cuts(cA, cB, lane, E.L, E.pp);
}

// The exact-T plans of degree pp (dp, tp fixed): every admissible microbatch
// count, largest first, gets its own split; a count whose lower bound (as in
// mem_counts, with the least slowest stage W of any split) lies past the tie
// window of the best time so far is not solved.  Plan slots, tallies and the
// returned least time as price_target.  The cut row of the cell's winner is
// rebuilt at the end of the cell.
template <int SLOTS, int S>
__device__ double price_exact(const BlockLds<SLOTS>& B, WaveLds& Wv, const double* U, int lane, int mv,
                              const JobCtx& jb, const TypeDev& ty, const Cell& cell, int tp, int pp, double W,
                              int& np, double best, double tie_eps, bool prune)
{
    const int dp = exact_quot(cell.n, tp * pp);
    const int grp = dp * tp;
    const double B_dp = link_bw(tiles_node(ty, grp), ty);
    bool adm = false;
    double b = 0.0;
    if (mv > 0) {
        // the nearest integer to Bg / (dp m) from a reciprocal estimate: exact
        // when dp m divides Bg, and the product test decides divisibility
        const double dm = (double)(dp * mv);
        const double q = rint((double)jb.Bg * rcp_approx(dm));
        adm = q * dm == (double)jb.Bg;
        b = q;
    }
    const unsigned long long amask = __ballot(adm);
    const int nadm = __popcll(amask);
    tally(Wv, lane, kAlgOps, 4ull * (unsigned)jb.L + (unsigned long long)nadm * (12ull * (unsigned)pp + 40ull));
    if (nadm == 0) return kInf;
    const int rank = __builtin_amdgcn_mbcnt_hi((unsigned)(amask >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)amask, 0u));
    if (adm) {
        Wv.bq[rank] = b;
        Wv.mq[rank] = mv;
    }
    wave_sync();
    const int base = np;
    np += nadm;
    if (np > kMaxPlans) {
        tally(Wv, lane, kOverflow, 1);
        np = kMaxPlans;
    }
    const double UL = U[jb.L * S];
    const double plb = fmax(B.Pp[jb.L] / (double)pp, B.p_layer_max);
    const double cP = dp > 1 ? cell.kappa * 2.0 * (double)(dp - 1) / (double)dp / ((double)tp * B_dp) : 0.0;
    double lim = prune ? best * (1.0 + tie_eps) : kInf;
    double best_t = kInf;
    for (int rk = nadm - 1; rk >= 0; --rk) {
        const double bm = Wv.bq[rk];
        const int m = Wv.mq[rk];
        double T = kInf;
        const double lbT = (bm * (UL + cell.c_p2p * ((double)(pp - 1) * B.x_layer_min)) + (double)(m - 1) * (bm * W) +
                            plb * cP) * (1.0 - 1e-9);
        if (!(lim < kInf) || lbT <= lim) {
            ExtCtx E;
            E.L = jb.L;
            E.pp = pp;
            E.m = m;
            E.b = bm;
            E.tpd = (double)tp;
            E.mem = ty.mem;
            E.cS = (double)(m - 1) * bm;
            E.cX = cell.kappa * 2.0 * bm / cell.B_pp;
            E.cP = cP;
            ExtKey key;
            if (ext_solve<S>(E, U, B.Pp, B.Ap, B.x, Wv.R, lane, key)) {
                // the stage costs sum to U_L; the cut-dependent rest is the key's Phi
                T = bm * UL + key.phi;
                best_t = fmin(best_t, T);
                if (prune) lim = fmin(lim, T * (1.0 + tie_eps));
            }
            tally(Wv, lane, kMemParts, 1);
        }
        if (lane == 0 && base + rk < kMaxPlans) {
            Wv.planT[base + rk] = T;
            Wv.planKey[base + rk] = ((unsigned)pp << 12) | ((unsigned)tp << 7) | (unsigned)m;
        }
        wave_sync();
    }
    return best_t;
}

// Price every admissible microbatch count of plan (dp, tp, pp) with the
// canonical stages of bottleneck W; appends to the wave's plan buffer.  Lane
// mi < n_m holds m_values[mi] (ascending) in `mv`: the lanes price one count
// each.  A stage's memory is non-increasing in m (min(m, pp-k) b is the batch
// share Bg/dp while m <= pp-k and falls after), so the counts that fit are the
// top of the admissible list; the first one is found by bisection.  Under
// the memory rule (MEM) each count below those, largest first, gets the
// balanced partition among the splits that fit (R: the wave's row for its
// recursion); counts stop once none fits (memory only grows as m falls) and,
// with `prune`, are skipped when a lower bound of their time lies past the
// tie window (tie_eps) of `best` or of a count priced here.  Returns the
// least time of the plans priced that fit (+inf if none): a plan of the
// cell, so an upper bound of the cell's best time.
template <int SLOTS, int S, bool MEM, bool EXT = false>
__device__ double price_target(BlockLds<SLOTS>& B, WaveLds& Wv, const double* U, int lane, int mv,
                               const JobCtx& jb, const TypeDev& ty, const Cell& cell, int tp, int pp,
                               double W, int& np, bool keep_cuts, double* R, double best, double tie_eps,
                               bool prune, uint8_t* pcache = nullptr)
{
    if constexpr (EXT) return price_exact<SLOTS, S>(B, Wv, U, lane, mv, jb, ty, cell, tp, pp, W, np, best, tie_eps,
                                                     prune);
    // S = 1: the pure-compute problem (U = Upure, W = Wtab[0][pp]), whose
    // splits the block keeps in pcache
    Stages sg;
    if constexpr (S == 1)
        sg = pp > 1 ? pure_split(U, W, B.pure_cached, Wv, pcache, lane, jb.L, pp)
                    : canonical_stages<1>(U, Wv.J, lane, jb.L, pp, W);
    else
        sg = canonical_stages<S>(U, Wv.J, lane, jb.L, pp, W);
    const int dp = exact_quot(cell.n, tp * pp);
    const int grp = dp * tp;
    const double B_dp = link_bw(tiles_node(ty, grp), ty);

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

    // lanes over the microbatch counts: admissible when dp m divides the batch
    // (the quotient of a correctly rounded division is exact then)
    bool adm = false;
    double b = 0.0;
    if (mv > 0) {
        // the nearest integer to Bg / (dp m) from a reciprocal estimate: exact
        // when dp m divides Bg, and the product test decides divisibility
        const double dm = (double)(dp * mv);
        const double q = rint((double)jb.Bg * rcp_approx(dm));
        adm = q * dm == (double)jb.Bg;
        b = q;
    }
    const unsigned long long amask = __ballot(adm);
    const int nadm = __popcll(amask);
    tally(Wv, lane, kAlgOps, 4ull * (unsigned)jb.L + (unsigned long long)nadm * (12ull * (unsigned)pp + 40ull));
    if (nadm == 0) return kInf;
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
    auto over_at = [&](int rk) {                            // does some stage overflow at rank rk?
        const double bm = Wv.bq[rk];
        const int m = Wv.mq[rk];
        const double i0 = (double)(m < r0 ? m : r0) * bm;
        const double i1 = (double)(m < r1 ? m : r1) * bm;
        const bool over = (act0 && fP0 + i0 * A0 > cap) || (act1 && fP1 + i1 * A1 > cap);
        return __ballot(over) != 0ull;
    };
    int lo = 0, hi = nadm;                                  // first fitting rank in [lo, hi]
    if constexpr (!MEM) {
        // a stage's memory falls as m grows: when the largest admissible count
        // does not fit, none does, and the degree's plans are priced infeasible
        // here (nothing of them enters the plan buffer)
        if (over_at(nadm - 1)) {
            tally(Wv, lane, kPlans, (unsigned long long)nadm);
            return kInf;
        }
        hi = nadm - 1;
    }
    // every count fits when the smallest does (the common case): one test
    if (lo < hi) {
        if (!over_at(0)) hi = 0; else lo = 1;
    }
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (!over_at(mid)) hi = mid; else lo = mid + 1;
    }

    double rs[1] = {sx}, rm[1] = {fmax(P0, P1)};
    wave_reduce<OpSum, 1>(rs);
    wave_reduce<OpMax, 1>(rm);
    const double sumX = rs[0];
    const double pmax = rm[0];
    const double sumS = U[jb.L * S];   // the stages tile the layers: sum of stage costs
    const double ar = (dp > 1)
        ? pmax * (cell.kappa * 2.0 * (double)(dp - 1) / ((double)dp * (double)tp * B_dp))
        : 0.0;
    const double per_sample = sumS + cell.c_p2p * sumX;   // fill time per sample

    double T = kInf;
    if (adm) {
        T = b * per_sample + (double)(mv - 1) * (b * W) + ar;
        const int slot = np + rank;
        if (slot < kMaxPlans) {
            Wv.planT[slot] = rank >= lo ? T : kInf;
            Wv.planKey[slot] = ((unsigned)pp << 12) | ((unsigned)tp << 7) | (unsigned)mv;
        }
    }
    const int base = np;
    np += nadm;
    if (np > kMaxPlans) {
        tally(Wv, lane, kOverflow, 1);
        np = kMaxPlans;
    }
    double best_t = kInf;
    if (lo < nadm) {
        best_t = bcast(T, 63 - __clzll(amask));   // the largest admissible count fits
        if (keep_cuts && best_t < Wv.cut_T) {
            // the cell's best time so far: keep this degree's cut row for the output
            if (lane < pp - 1) Wv.cutrow[lane] = (uint8_t)sg.hi0;
            if (lane + 64 < pp - 1) Wv.cutrow[lane + 64] = (uint8_t)sg.hi1;
            if (lane == 0) {
                Wv.cut_T = best_t;
                Wv.cut_tp = tp;
                Wv.cut_pp = pp;
                Wv.cut_m = 0;
                Wv.cut_mfit = Wv.mq[lo];
            }
        }
    }
    if constexpr (MEM) {
        if (lo > 0) {
            wave_sync();
            const double c_ar = (dp > 1) ? cell.kappa * 2.0 * (double)(dp - 1) / ((double)dp * (double)tp * B_dp)
                                         : 0.0;
            best_t = mem_counts<S>((const Lds<double>*)U, (const Lds<double>*)B.Pp, (const Lds<double>*)B.Ap,
                                   (const Lds<float>*)B.x, (Lds<double>*)R, (Lds<WaveLds>*)&Wv, lane, jb.L, tp, pp,
                                   dp, lo, base, W, cap, sumS,
                                   cell.c_p2p, c_ar, fmax(B.Pp[jb.L] / (double)pp, B.p_layer_max), B.x_layer_min,
                                   best_t, prune ? fmin(best, best_t) * (1.0 + tie_eps) : kInf, tie_eps, prune,
                                   keep_cuts);
        }
    }
    return best_t;
}


// What the lower bounds of one problem's plans share: its tensor degree, n /
// tp, a lower bound of its summed per-sample layer costs, and the gradient
// all-reduce seconds per parameter byte over the intra- and inter-node links
// without the ring factor (kappa 2 / (tp B)).
struct BoundCtx {
    int tp, qn;
    double rtp;
    double UL;
    double ar_intra, ar_inter;
    double cx, cq;                // seconds per sample per x byte and per all-to-all byte of a layer
};

// Lower bound of the iteration time of every plan of degree pp (any listed m)
// of problem bc, or +inf when no split of the layers into pp stages fits
// memory.  Bounded below without the cuts:
//   W*(pp) >= UL / pp (the stages tile the layers), and the stage of the
//   optimal split whose pure-compute cost is largest reaches Wpure(pp) (no
//   split of pp stages does better), so it is a window of layers reaching
//   Wpure(pp): W*(pp) >= Wpure(pp) / tp + cx xwin(pp) + cq qwin(pp);
//   the p2p bytes over the pp-1 stage boundaries >= (pp-1) min_l x_l;
//   the largest stage's parameters >= max(P / pp, max_l p_l).
// Memory: besides the parameter bound, the stage holding layer l has at most
// l - 1 stages before it, so at least min(m, pp - l + 1) microbatches in
// flight; for l = 1, 2, that layer's own bytes with that many microbatches at
// the largest admissible m lower-bound the pricing's test of that stage term
// by term (prefix differences, exact integer counts), so when they overflow,
// no split fits with any m (memory falls as m grows).
// For fixed dp, T = Bg/dp W + Bg/(dp m) (fill - W) + AR falls as m grows
// (fill >= W), so the largest admissible m gives the bound.  Reciprocals are
// estimates; a relative margin of 1e-9 covers them and the rounding.
template <int SLOTS>
__device__ double target_bound(const BlockLds<SLOTS>& B, const JobCtx& jb, const TypeDev& ty, const Cell& cell,
                               unsigned gpn_divs, BoundCtx bc, int pp)
{
    const double rpp = rcp_approx((double)pp);
    const int dp = (int)rint((double)bc.qn * rpp);                     // exact: pp divides qn
    const int m = B.mmax[dp - 1];
    const double plb = fmax(B.Pp[jb.L] * rpp, B.p_layer_max);
    if (4.0 * plb > ty.mem * (double)bc.tp * (1.0 + 1e-9)) return kInf;
    const double b = rint((double)jb.Bg * rcp_approx((double)(dp * m)));   // exact: dp m divides Bg
    {
        const double cap = ty.mem * (double)bc.tp;
        bool over = false;
#pragma unroll
        for (int l = 1; l <= kHeadLayers; ++l) {
            const int r = pp - l + 1;
            const int f = m < r ? m : (r > 1 ? r : 1);
            over |= 4.0 * B.head_p[l - 1] + (double)f * b * B.head_a[l - 1] > cap;
        }
        if (over) return kInf;
    }
    const double Wlb = fmax(bc.UL * rpp, B.Wtab[0][pp] * bc.rtp + (bc.cx * (double)B.xwin[pp] +
                                                                    bc.cq * (double)B.qwin[pp]));
    const double fill = bc.UL + cell.c_p2p * ((double)(pp - 1) * B.x_layer_min);
    const int grp = dp * bc.tp;
    const double c_ar = (grp < 32 && ((gpn_divs >> grp) & 1u)) ? bc.ar_intra : bc.ar_inter;
    const double ar = dp > 1 ? plb * (c_ar * ((double)(dp - 1) * rcp_approx((double)dp))) : 0.0;
    return (b * fill + (double)(m - 1) * (b * Wlb) + ar) * (1.0 - 1e-9);
}

// Lower bounds of the degrees in `tm` into Wv.lbnd[pp - 1], one lane per
// degree (a problem requests at most 32 degrees: the divisors of n / tp);
// returns the least of them (+inf: no degree fits memory).
template <int SLOTS>
__device__ __forceinline__ double degree_bounds(const BlockLds<SLOTS>& B, WaveLds& Wv, const Mask& tm, int lane,
                                                const JobCtx& jb, const TypeDev& ty, const Cell& cell,
                                                unsigned gpn_divs, const BoundCtx& bc)
{
    const bool b0 = (tm.lo >> lane) & 1ull, b1 = (tm.hi >> lane) & 1ull;
    const unsigned r0 = __builtin_amdgcn_mbcnt_hi((unsigned)(tm.lo >> 32),
                                                  __builtin_amdgcn_mbcnt_lo((unsigned)tm.lo, 0u));
    const unsigned r1 = (unsigned)__popcll(tm.lo) +
                        __builtin_amdgcn_mbcnt_hi((unsigned)(tm.hi >> 32),
                                                  __builtin_amdgcn_mbcnt_lo((unsigned)tm.hi, 0u));
    if (b0 && r0 < 64u) Wv.tq[r0] = (uint8_t)(1 + lane);
    if (b1 && r1 < 64u) Wv.tq[r1] = (uint8_t)(65 + lane);
    wave_sync();
    double lb = kInf;
    if (lane < tm.count()) {
        const int pp = Wv.tq[lane];
        lb = target_bound(B, jb, ty, cell, gpn_divs, bc, pp);
        Wv.lbnd[pp - 1] = lb;
    }
    wave_sync();
    return wave_reduce1<OpMin>(lb);
}

// The bound context of the cell's problem of tensor degree tp; the pure-
// compute problem (tp = 1 without all-to-all) takes its exact cost sum.
__device__ __forceinline__ BoundCtx bound_ctx(const Cell& cell, int tp, double UL, double ar_intra1,
                                              double ar_inter1, double cx1 = 0.0, double cq = 0.0)
{
    BoundCtx bc;
    bc.tp = tp;
    bc.qn = exact_quot(cell.n, tp);
    bc.rtp = tp == 1 ? 1.0 : rcp_approx((double)tp);
    bc.UL = UL;
    bc.ar_intra = ar_intra1 * bc.rtp;
    bc.ar_inter = ar_inter1 * bc.rtp;
    bc.cx = cx1 * ((double)(tp - 1) * bc.rtp);
    bc.cq = cq;
    return bc;
}

// Slot of the shared problem (tp, variant), -1 if the cell solves its own.
template <int SLOTS>
__device__ __forceinline__ int find_slot(const BlockLds<SLOTS>& B, int n_slots, bool moe, int tp, int var)
{
    if (tp == 1 && (var == 1 || !moe)) return 0;
    int slot = -1;
    for (int s = 1; s < n_slots; ++s)
        if (B.slot_tp[s] == tp && B.slot_var[s] == var) slot = s;
    return slot;
}

// Inclusive prefix sum over the wave (row shifts, then row broadcasts): the
// order of the additions is a tree's, which is all a bound needs.
__device__ __forceinline__ double wave_incl_sum(double v)
{
    v += dpp<0x111, 0xf>(v, 0.0);   // row_shr:1
    v += dpp<0x112, 0xf>(v, 0.0);   // row_shr:2
    v += dpp<0x114, 0xf>(v, 0.0);   // row_shr:4
    v += dpp<0x118, 0xf>(v, 0.0);   // row_shr:8
    v += dpp<0x142, 0xa>(v, 0.0);   // row_bcast:15 into rows 1 and 3
    v += dpp<0x143, 0xc>(v, 0.0);   // row_bcast:31 into rows 2 and 3
    return v;
}

// For every degree pp <= L: the least x bytes and the least all-to-all bytes
// of a window of consecutive layers whose pure-compute cost (a difference of
// Upure, as the recursion forms it) reaches Wtab[0][pp], rounded down with a
// relative margin for the sums' rounding.  The waves share the degrees; the
// x and all-to-all prefixes sit in each wave's UD (x even, all-to-all odd).
template <int SLOTS>
__device__ void window_minima(BlockLds<SLOTS>& B, WaveLds& Wv, int lane, int wid, int L, const float* xg,
                              const float* qg, bool moe)
{
    double* P = Wv.UD;
    const double x0 = lane < L ? (double)xg[lane] : 0.0, x1 = lane + 64 < L ? (double)xg[lane + 64] : 0.0;
    // without all-to-all layers every q is 0 and so is every window's
    const double q0 = moe && lane < L ? (double)qg[lane] : 0.0, q1 = moe && lane + 64 < L ? (double)qg[lane + 64] : 0.0;
    const double sx0 = wave_incl_sum(x0), sq0 = wave_incl_sum(q0);
    const double tx = bcast(sx0, 63), tq = bcast(sq0, 63);
    const double sx1 = wave_incl_sum(x1) + tx, sq1 = wave_incl_sum(q1) + tq;
    if (lane == 0) {            // zero (lane 0's sum is its own value), kept out of a constant register
        P[0] = sx0 - x0;
        P[1] = sq0 - q0;
    }
    if (lane < L) {
        P[2 * (lane + 1)] = sx0;
        P[2 * (lane + 1) + 1] = sq0;
    }
    if (lane + 64 < L) {
        P[2 * (lane + 65)] = sx1;
        P[2 * (lane + 65) + 1] = sq1;
    }
    wave_sync();
    const double* U = B.Upure;
    // the bottlenecks fall as pp grows (a split refines into one more stage), so
    // a start's first reaching end does too: each search ends at the last one
    int end[2] = {L, L};
    for (int pp = wid + 1; pp <= L; pp += kWavesPerBlock) {
        const double th = B.Wtab[0][pp];
        double bx = kInf, bq = kInf;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int i = lane + 64 * h;
            if (i < L) {
                const double Ui = U[i];
                if (U[L] - Ui >= th) {
                    int lo = i + 1, hi = end[h];    // the first end whose window reaches th
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (U[mid] - Ui >= th) hi = mid; else lo = mid + 1;
                    }
                    end[h] = lo;
                    bx = fmin(bx, P[2 * lo] - P[2 * i]);
                    if (moe) bq = fmin(bq, P[2 * lo + 1] - P[2 * i + 1]);
                }
            }
        }
        bx = wave_reduce1<OpMin>(bx);
        if (moe) bq = wave_reduce1<OpMin>(bq);
        if (lane == 0) {
            B.xwin[pp] = __double2float_rd(fmax(bx, 0.0) * (1.0 - 1e-9));
            B.qwin[pp] = moe ? __double2float_rd(fmax(bq, 0.0) * (1.0 - 1e-9)) : 0.0f;
        }
    }
}

// ------------------------------------------------------------ the kernel

// A block's work tallies live in its waves' LDS for the whole launch: zeroed
// before its first item and added to the device counters once, after its
// last (a device-wide atomic per item and counter would cost HBM writes).
constexpr int kZeroTallies = -2;
constexpr int kFlushTallies = -1;

__device__ __forceinline__ void block_tallies(const EstimateArgs& A, WaveLds& Wv, int lane, int op)
{
    if (op == kZeroTallies) {
        if (lane < kNumCounters) Wv.tally[lane] = 0ull;
        wave_sync();
        return;
    }
    if (lane == 0) {
        const unsigned long long* t = Wv.tally;
        for (int c = 0; c < kNumCounters; ++c) {
            const unsigned long long v = c == kAlgOps ? t[kAlgOps] + 8ull * t[kDpEntries] : t[c];
            if (v) atomicAdd(&A.counters[c], v);
        }
    }
}

// MEM: the memory-constrained partition rule (each wave has one more LDS
// row for its recursion); EXT: the exact-T rule (that row holds its
// suffix recursion).
template <int SLOTS, bool MEM, bool EXT = false>
__device__ __forceinline__ void estimate_body(const EstimateArgs& A, int wid, int item)
{
    __shared__ BlockLds<SLOTS> B;
    // the wave index (wid) is taken once per launch, as a scalar; the lane
    // index (counted by mbcnt, not kept from the launch) passes through an
    // empty asm statement once per item, so nothing derived from it is hoisted
    // out of the item loop and held in registers across every item (it would
    // be spilled)
    int lane0;
    __asm__ volatile("" : "=v"(lane0) : "0"((int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u))));
    const int lane = lane0;
    const int tid = wid * 64 + lane;
    WaveLds& Wv = B.w[wid];
    double* const R = MEM ? Wv.R : nullptr;
    if (item < 0) {
        block_tallies(A, Wv, lane, item);
        return;
    }
    uint8_t* const pcache = A.pure_cuts + (size_t)blockIdx.x * kPureCutBytes;

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
    const unsigned gpn_divs = ty.divs;   // bit d: d divides the node size

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
        seq_prefix<1, 2>(v0, v1, jb.L, lane, wid == 0 ? B.Pp : B.Ap, Wv.UD + 1, false);
        if (wid == 0) {
            const double pm = wave_reduce1<OpMax>(fmax(v0, v1));
            if (lane == 0) B.p_layer_max = pm;
        }
    } else if (wid == 2) {
        build_prefix_u<1>(B.t, B.x, B.q, B.Upure, Wv.UD + 1, lane, jb, ty, 1.0, 1, false);
    } else {
        bool same = true;
        for (int c = lane; c < A.n_counts; c += 64) same &= A.kappa[g * A.n_counts + c] == A.kappa[g * A.n_counts];
        const bool uni = __ballot(!same) == 0ull;
        const double x0 = lane < jb.L ? (double)A.x[off + lane] : kInf;
        const double x1 = lane + 64 < jb.L ? (double)A.x[off + lane + 64] : kInf;
        const double xm = wave_reduce1<OpMin>(fmin(x0, x1));
        const double xs = wave_reduce1<OpSum>((lane < jb.L ? (double)A.x[off + lane] : 0.0) +
                                              (lane + 64 < jb.L ? (double)A.x[off + lane + 64] : 0.0));
        const double qs = wave_reduce1<OpSum>((lane < jb.L ? (double)A.q[off + lane] : 0.0) +
                                              (lane + 64 < jb.L ? (double)A.q[off + lane + 64] : 0.0));
        if (lane == 0) {
            B.x_sum = xs;
            B.q_sum = qs;
            B.uniform = uni ? 1 : 0;
            B.next_cell = 0;
            B.moe = jb.moe ? 1 : 0;
            B.x_layer_min = xm;
            B.pure_cached[0] = 0ull;
            B.pure_cached[1] = 0ull;
        }
    }
    // largest admissible microbatch count of each data-parallel degree.  Below
    // 2^20 samples the quotients come from float reciprocals (relative error
    // about 2^-23, so rounding gives the exact quotient of a divisor) and a
    // product check decides divisibility; larger batches take integer remainders.
    const bool small_batch = jb.Bg < (1 << 20);
    for (int dp = tid + 1; dp <= kMaxDp; dp += 256) {
        int mm = 0, mc = 0;
        if (small_batch) {
            const int q = (int)rintf((float)jb.Bg * __builtin_amdgcn_rcpf((float)dp));
            if (q * dp == jb.Bg) {
                for (int i = 0; i < A.n_m; ++i) {
                    const int m = A.m_values[i];
                    const int r = (int)rintf((float)q * __builtin_amdgcn_rcpf((float)m));
                    if (r * m == q) {
                        mm = m > mm ? m : mm;
                        ++mc;
                    }
                }
            }
        } else {
            for (int i = 0; i < A.n_m; ++i)
                if (jb.Bg % (dp * A.m_values[i]) == 0) {
                    mm = A.m_values[i] > mm ? A.m_values[i] : mm;
                    ++mc;
                }
        }
        B.mmax[dp - 1] = (uint8_t)mm;
        B.mcnt[dp - 1] = (uint8_t)mc;
    }
    __syncthreads();

    // ---- shared problems: the pure-compute one (every degree up to L: its
    // bottlenecks also bound the other problems'), and every tensor degree
    // when the type's contention factor is the same for all counts
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
    if (tid < kHeadLayers) {
        B.head_p[tid] = tid < jb.L ? B.Pp[tid + 1] - B.Pp[tid] : 0.0;
        B.head_a[tid] = tid < jb.L ? B.Ap[tid + 1] - B.Ap[tid] : 0.0;
    }
    if (wid == 0) tally(Wv, lane, kCells, (unsigned long long)A.n_counts);

    for (int s = wid; s < n_slots; s += kWavesPerBlock) {
        const int tp = B.slot_tp[s], var = B.slot_var[s];
        Mask tm;
        if (s == 0) {
            tm = ballot_mask(1 + lane <= jb.L, 65 + lane <= jb.L);
        } else {
            bool ok0 = false, ok1 = false;
            for (int c = 0; c < A.n_counts; ++c) {
                const int n = A.counts[c];
                if (n % tp != 0) continue;
                ok0 |= target_ok(B.mmax, jb, n, tp, var, 1 + lane);
                ok1 |= target_ok(B.mmax, jb, n, tp, var, 65 + lane);
            }
            tm = ballot_mask(ok0, ok1);
        }
        if (!tm.any()) continue;
        if (s > 0) {
            build_prefix_u<2>(B.t, B.x, B.q, Wv.UD, Wv.UD + 1, lane, jb, ty, (double)A.kappa[g * A.n_counts],
                              tp, true);
        } else {
            for (int e = lane; e < kLmax + kPad; e += 64) Wv.UD[2 * e] = B.Upure[e];
            wave_sync();
        }
        double* Wrow = B.Wtab[s];
        solve_dp(Wv, jb.L, tm, lane, [&](int pp, double W, Mask m) {
            if (lane == 0) Wrow[pp] = W;
            return m;
        });
        tally(Wv, lane, kProblems, 1);
        tally(Wv, lane, kAlgOps, 8ull * (unsigned)jb.L);
    }
    __syncthreads();
    window_minima(B, Wv, lane, wid, jb.L, A.x + off, A.q + off, jb.moe);
    __syncthreads();

    // ---- cells: take counts, largest first, from the block's work counter
    for (;;) {
        // the lane index is re-derived per cell, for the same reason as the
        // thread index per item
        int lane;
        __asm__ volatile("" : "=v"(lane) : "0"((int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u))));
        int cix = 0;
        if (lane == 0) cix = atomicAdd(&B.next_cell, 1);
        cix = __builtin_amdgcn_readfirstlane(cix);
        if (cix >= A.n_counts) break;
        const int ci = A.count_order[cix];
        Cell cell;
        cell.n = A.counts[ci];
        cell.kappa = (double)A.kappa[g * A.n_counts + ci];
        cell.B_pp = link_bw(cell.n <= ty.gpn, ty);
        cell.c_p2p = cell.kappa * 2.0 / cell.B_pp;
        int np = 0;
        double best = kInf;          // time of a fitting plan priced so far: bounds the cell's best
        if (lane == 0) Wv.cut_T = kInf;
        // per-cell pieces of the bounds: all-reduce seconds per byte (tp = 1),
        // and the tensor-parallel and all-to-all parts of a problem's cost sum.
        // Bounds only: their relative margins cover reciprocal estimates (the
        // memory rule's kernel keeps the divisions, which measured faster there);
        // a bandwidth of +inf (no such link) gives 0, as the division does
        auto bdiv = [](double x, double y) {
            if constexpr (MEM) return x / y;
            else return y < kInf ? x * rcp_approx(y) : 0.0;
        };
        const double ar_intra1 = bdiv(cell.kappa * 2.0, ty.bw_intra);
        const double ar_inter1 = bdiv(cell.kappa * 2.0, ty.bw_inter);
        const double ul_tp = bdiv(cell.kappa * 8.0 * B.x_sum, ty.bw_intra);
        const double ul_a2a = jb.moe ? bdiv(cell.kappa * B.q_sum, ty.bw_inter) : 0.0;
        // per byte of a layer: tensor-parallel seconds (times (tp-1)/tp) and all-to-all seconds
        const double cx1 = bdiv(cell.kappa * 8.0, ty.bw_intra);
        const double cq1 = jb.moe ? bdiv(cell.kappa, ty.bw_inter) : 0.0;

        // plans of the pure-compute problem first: their bottlenecks are shared
        {
            const int var = jb.moe ? 1 : 0;
            const Mask tm = ballot_mask(target_ok(B.mmax, jb, cell.n, 1, var, 1 + lane),
                                        target_ok(B.mmax, jb, cell.n, 1, var, 65 + lane));
            if (tm.any()) {
                // bounds with the exact bottleneck; a degree is priced unless its
                // bound is past the tie window of the best plan so far
                degree_bounds(B, Wv, tm, lane, jb, ty, cell, gpn_divs,
                              bound_ctx(cell, 1, B.Upure[jb.L], ar_intra1, ar_inter1));
                for (int pp = tm.next(1); pp; pp = tm.next(pp + 1)) {
                    const double lbp = Wv.lbnd[pp - 1];
                    if (A.prune && !(lbp < kInf && lbp <= best * (1.0 + A.tie_eps))) continue;
                    best = fmin(best, price_target<SLOTS, 1, MEM, EXT>(B, Wv, B.Upure, lane, mv, jb, ty, cell, 1, pp,
                                                                  B.Wtab[0][pp], np, A.cuts != nullptr, R, best,
                                                                  A.tie_eps, A.prune != 0, pcache));
                }
            }
        }
        // the other problems, best first: every tensor degree's problem gets the
        // least lower bound of its plans, then the problem of least bound is
        // solved while that bound lies within the tie window of `best` (so the
        // first problem solved is the most promising one and its plans tighten
        // the window for the rest).  Within a problem a degree whose bound
        // exceeds the window cannot hold the cell's plan and is skipped, and the
        // recursion stops after the last degree still wanted.
        const int tpmax = cell.n < ty.gpn ? cell.n : ty.gpn;
        int ncand = 0;
        for (int tp = 1; tp <= tpmax; ++tp) {
            if (((gpn_divs >> tp) & 1u) == 0 || exact_quot(cell.n, tp) * tp != cell.n) continue;
            if (tp == 1 && !jb.moe) continue;          // the pure-compute problem
            const Mask tm = ballot_mask(target_ok(B.mmax, jb, cell.n, tp, 0, 1 + lane),
                                        target_ok(B.mmax, jb, cell.n, tp, 0, 65 + lane));
            if (!tm.any()) continue;
            // the layer costs sum to at least this (the job's sums of x and of the
            // all-to-all bytes in the cost formula; margin for the rounding)
            const double rtp = tp == 1 ? 1.0 : rcp_approx((double)tp);
            const double ULb = ((B.Upure[jb.L] + (double)(tp - 1) * ul_tp) * rtp + ul_a2a) * (1.0 - 1e-12);
            const double lb = degree_bounds(B, Wv, tm, lane, jb, ty, cell, gpn_divs,
                                            bound_ctx(cell, tp, ULb, ar_intra1, ar_inter1, cx1, cq1));
            if (lane == 0) {
                Wv.cand_tp[ncand] = (uint8_t)tp;
                Wv.cand_lb[ncand] = lb;
            }
            ++ncand;
        }
        wave_sync();
        unsigned solved = 0;           // bit c: candidate c has been taken
        for (;;) {
            int csel = -1;
            double lsel = kInf;
            for (int c = 0; c < ncand; ++c) {
                const double v = Wv.cand_lb[c];
                if (!((solved >> c) & 1u) && (csel < 0 || v < lsel)) {
                    csel = c;
                    lsel = v;
                }
            }
            if (csel < 0) break;
            if (A.prune && !(lsel < kInf && lsel <= best * (1.0 + A.tie_eps))) break;
            // the first problem taken, if it is the last one bounded above, still has
            // its degrees' bounds in lbnd (tp ascending: the largest tp, whose
            // problem is most often taken first on the full round, is bounded last)
            const bool fresh = solved == 0u && csel == ncand - 1;
            solved |= 1u << csel;
            const int tp = Wv.cand_tp[csel];
            Mask tm = ballot_mask(target_ok(B.mmax, jb, cell.n, tp, 0, 1 + lane),
                                  target_ok(B.mmax, jb, cell.n, tp, 0, 65 + lane));
            if (!fresh) {
                const double rtp = tp == 1 ? 1.0 : rcp_approx((double)tp);
                const double ULb = ((B.Upure[jb.L] + (double)(tp - 1) * ul_tp) * rtp + ul_a2a) * (1.0 - 1e-12);
                degree_bounds(B, Wv, tm, lane, jb, ty, cell, gpn_divs,
                              bound_ctx(cell, tp, ULb, ar_intra1, ar_inter1, cx1, cq1));
            }
            // kept: no bound yet (+inf: memory rules the degree out), or within the window
            {
                const double lb0 = Wv.lbnd[lane], lb1 = Wv.lbnd[lane + 64];
                const double lim = best * (1.0 + A.tie_eps);
                if (A.prune) tm = tm & ballot_mask(lb0 < kInf && lb0 <= lim, lb1 < kInf && lb1 <= lim);
            }
            if (!tm.any()) continue;
            double u[2];
            layer_costs(B.t, B.x, B.q, lane, jb, ty, cell.kappa, tp, true, u);
            seq_prefix<2, 2>(u[0], u[1], jb.L, lane, Wv.UD, Wv.UD + 1, true);
            tally(Wv, lane, kAlgOps, 8ull * (unsigned)jb.L);
            const int slot = find_slot(B, n_slots, jb.moe, tp, 0);
            if (slot > 0) {
                for (int pp = tm.next(1); pp; pp = tm.next(pp + 1)) {
                    const double lbp = Wv.lbnd[pp - 1];
                    if (A.prune && !(lbp <= best * (1.0 + A.tie_eps))) continue;
                    best = fmin(best, price_target<SLOTS, 2, MEM, EXT>(B, Wv, Wv.UD, lane, mv, jb, ty, cell, tp, pp,
                                                                  B.Wtab[slot][pp], np, A.cuts != nullptr, R, best,
                                                                  A.tie_eps, A.prune != 0));
                }
            } else {
                // prices degree pp at bottleneck W; returns the degrees still wanted
                auto price_deg = [&](int pp, double W, Mask m) -> Mask {
                    best = fmin(best, price_target<SLOTS, 2, MEM, EXT>(B, Wv, Wv.UD, lane, mv, jb, ty, cell, tp, pp, W,
                                                                  np, A.cuts != nullptr, R, best, A.tie_eps,
                                                                  A.prune != 0));
                    const double lim = best * (1.0 + A.tie_eps);
                    Mask rest = m;                       // degrees still to come
                    if (pp <= 64) rest.lo &= ~(1ull << (pp - 1)); else rest.hi &= ~(1ull << (pp - 65));
                    return A.prune ? rest & ballot_mask(Wv.lbnd[lane] <= lim, Wv.lbnd[lane + 64] <= lim) : rest;
                };
                // the largest requested degrees first: where a certificate gives the
                // bottleneck, the recursion is spared their rows (not under the
                // exact-T rule, whose pricing outweighs its few recursions: taken
                // largest first it prices more plans than it saves rows)
                if constexpr (!EXT) {
                    for (int pc = tm.last(); pc >= kCertMinDegree; pc = tm.last()) {
                        // the memory test of the degree's largest admissible count
                        // (not under the memory rule, whose splits differ)
                        const int dpc = exact_quot(cell.n, tp * pc);
                        double wc;
                        if constexpr (MEM) {
                            wc = certified_bottleneck<2>(
                                pure_split(B.Upure, B.Wtab[0][pc], B.pure_cached, Wv, pcache, lane, jb.L, pc), Wv,
                                lane, jb.L, pc);
                        } else {
                            const int mx = B.mmax[dpc - 1];
                            const double bmx = rint((double)jb.Bg * rcp_approx((double)(dpc * mx)));   // exact
                            wc = certified_bottleneck<kCertRounds, true>(
                                pure_split(B.Upure, B.Wtab[0][pc], B.pure_cached, Wv, pcache, lane, jb.L, pc), Wv,
                                lane, jb.L, pc, B.Pp, B.Ap, ty.mem * (double)tp, bmx, mx < pc ? mx : pc);
                        }
                        if (wc == -2.0) {
                            // no count fits: its plans are priced infeasible without the bottleneck
                            tally(Wv, lane, kPlans, (unsigned long long)B.mcnt[dpc - 1]);
                            if (pc <= 64) tm.lo &= ~(1ull << (pc - 1)); else tm.hi &= ~(1ull << (pc - 65));
                            continue;
                        }
                        if (!(wc >= 0.0)) break;
                        tm = price_deg(pc, wc, tm);
                    }
                }
                if (tm.any()) {
                    solve_dp(Wv, jb.L, tm, lane, price_deg);
                    tally(Wv, lane, kProblems, 1);
                }
            }
        }
        wave_sync();

        // best plan of the cell: smallest key among plans within the tie window
        double tl = kInf;
        for (int e = lane; e < np; e += 64) tl = fmin(tl, Wv.planT[e]);
        const double tmin = wave_reduce1<OpMin>(tl);
        const long long cidx = ((long long)j * A.n_types + g) * A.n_counts + ci;
        tally(Wv, lane, kPlans, (unsigned long long)np);
        if (!(tmin < kInf)) {
            tally(Wv, lane, kInfeasible, 1);
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
        const double tlim = tmin * (1.0 + A.tie_eps);
        // the smallest key within the window and its entry in one reduction
        // (keys are unique in a cell; key 256 + entry < 2^28 is exact)
        double kl = kInf;
        for (int e = lane; e < np; e += 64)
            if (Wv.planT[e] <= tlim) kl = fmin(kl, (double)Wv.planKey[e] * 256.0 + (double)e);
        const double kv = wave_reduce1<OpMin>(kl);
        const unsigned kbest = (unsigned)(kv * (1.0 / 256.0));
        int ib = (int)(kv - (double)kbest * 256.0);
        ib = ib < 0 ? 0 : (ib >= np ? np - 1 : ib);
        const double Tb = Wv.planT[ib];
        const int pp = (int)(kbest >> 12);
        const int tp = (int)((kbest >> 7) & 0x1Fu);
        const int m = (int)(kbest & 0x7Fu);
        const int dp = exact_quot(cell.n, tp * pp);
        if (lane == 0) {
            const float tt = (float)Tb, th = (float)((double)jb.Bg / Tb);
            const uint32_t pw = (unsigned)dp | ((unsigned)tp << 11) | ((unsigned)pp << 16) |
                                ((unsigned)m << 24) | (1u << 31);
            A.t_iter[cidx] = tt;
            A.thr[cidx] = th;
            A.plan[cidx] = pw;
        }
        const bool kept = !EXT && Wv.cut_tp == tp && Wv.cut_pp == pp && Wv.cut_T < kInf &&
                          (!MEM || (Wv.cut_m == 0 ? m >= Wv.cut_mfit : Wv.cut_m == m));
        if (A.cuts && kept) {
            // the winner is the plan kept while pricing (balanced cuts depend on
            // tp and pp only; memory-rule cuts also on m)
            uint8_t* row = A.cuts + cidx * A.cuts_stride;
            for (int e = lane; e < A.cuts_stride; e += 64)
                row[e] = (e < pp - 1) ? Wv.cutrow[e] : (uint8_t)0xFF;
        } else if (A.cuts) {
            // re-derive the winner's bottleneck and cuts
            const int var = (jb.moe && dp * tp == 1) ? 1 : 0;
            const int slot = find_slot(B, n_slots, jb.moe, tp, var);
            const double* U = Wv.UD;
            if (slot == 0) {
                for (int e = lane; e < kLmax + kPad; e += 64) Wv.UD[2 * e] = B.Upure[e];
                wave_sync();
            } else {
                build_prefix_u<2>(B.t, B.x, B.q, Wv.UD, Wv.UD + 1, lane, jb, ty, cell.kappa, tp, var == 0);
            }
            double W = 0.0;
            if (slot >= 0) {
                W = B.Wtab[slot][pp];
            } else {
                Mask one;
                one.lo = pp <= 64 ? (1ull << (pp - 1)) : 0ull;
                one.hi = pp > 64 ? (1ull << (pp - 65)) : 0ull;
                const unsigned long long e0 = Wv.tally[kDpEntries];   // the cuts' rerun is not tallied
                solve_dp(Wv, jb.L, one, lane, [&](int, double Wk, Mask mk) {
                    W = Wk;
                    return mk;
                });
                if (lane == 0) Wv.tally[kDpEntries] = e0;
            }
            Stages sg;
            if constexpr (EXT) {
                // the winner's exact-T split, solved again for its count
                const double bw = rint((double)jb.Bg / (double)(dp * m));
                const int grp = dp * tp;
                const double B_dp = link_bw(tiles_node(ty, grp), ty);
                ExtCtx E;
                E.L = jb.L;
                E.pp = pp;
                E.m = m;
                E.b = bw;
                E.tpd = (double)tp;
                E.mem = ty.mem;
                E.cS = (double)(m - 1) * bw;
                E.cX = cell.kappa * 2.0 * bw / cell.B_pp;
                E.cP = dp > 1 ? cell.kappa * 2.0 * (double)(dp - 1) / (double)dp / ((double)tp * B_dp) : 0.0;
                ExtKey key;
                ext_solve<2>(E, U, B.Pp, B.Ap, B.x, Wv.R, lane, key);
                sg = ext_cuts<2>(E, U, B.Pp, B.Ap, B.x, Wv.R, lane, key);
            } else {
                sg = canonical_stages<2>(U, Wv.J, lane, jb.L, pp, W);
            }
            if constexpr (MEM) {
                // the balanced split if it fits with the winner's m, else the rule's
                const double dm = (double)(dp * m);
                const double bw = rint((double)jb.Bg / dm);
                const double cap = ty.mem * (double)tp;
                if (!stages_fit(sg, B.Pp, B.Ap, lane, pp, m, bw, cap)) {
                    unsigned ent = 0;
                    const double Wm = mem_bottleneck<2>(U, B.Pp, B.Ap, R, lane, jb.L, pp, m, bw, cap, ent);
                    mem_cuts<2>(U, B.Pp, B.Ap, lane, jb.L, pp, m, bw, cap, Wm, sg);
                }
            }
            uint8_t* row = A.cuts + cidx * A.cuts_stride;
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const int idx = lane + 64 * s;
                const int en = s == 0 ? +sg.hi0 : +sg.hi1;
                if (idx < A.cuts_stride) row[idx] = (idx < pp - 1) ? (uint8_t)en : (uint8_t)0xFF;
            }
            for (int e = 128 + lane; e < A.cuts_stride; e += 64) row[e] = 0xFF;
        }
        wave_sync();
    }
}

// The (job, type) item a block works on next.  The host deals whole jobs to
// kQueues queues of about equal work, heaviest first, with the items of one
// job adjacent; a block takes the next item of the queue of its XCD
// (workgroups are handed to the XCDs round robin, so block b runs on XCD
// b mod 8), so the types of one job run on one XCD and its layer tables are
// fetched into that XCD's L2 once.  A block whose queue is empty takes from
// the next queues in turn, so the work still balances over every CU whatever
// the items really cost.  Returns the item, or -1 once every queue is empty
// (every block then leaves).
__device__ __forceinline__ int take_item(const EstimateArgs& A, int* slot, int wid)
{
    if (wid == 0 && __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) == 0u) {
        int item = -1;
        for (int r = 0; r < kQueues && item < 0; ++r) {
            const int qi = (int)((blockIdx.x + r) % kQueues);
            const unsigned long long len = (unsigned long long)(A.queue_off[qi + 1] - A.queue_off[qi]);
            if (len == 0ull) continue;
            const unsigned long long q = atomicAdd(&A.queue[qi], 1ull);
            if (q < len) item = A.item_order[A.queue_off[qi] + (int)q];
        }
        *slot = item;
    }
    __syncthreads();
    const int item = *slot;
    __syncthreads();
    return item;
}

template <int SLOTS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void estimate_kernel(EstimateArgs A)
{
    __shared__ int slot;
    const int wid = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    estimate_body<SLOTS, false>(A, wid, kZeroTallies);
    for (int item = take_item(A, &slot, wid); item >= 0; item = take_item(A, &slot, wid)) {
        estimate_body<SLOTS, false>(A, wid, item);
        __syncthreads();
    }
    estimate_body<SLOTS, false>(A, wid, kFlushTallies);
}

// The exact-T rule: each plan's split minimises its iteration time.
template <int SLOTS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void estimate_ext_kernel(EstimateArgs A)
{
    __shared__ int slot;
    const int wid = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    estimate_body<SLOTS, false, true>(A, wid, kZeroTallies);
    for (int item = take_item(A, &slot, wid); item >= 0; item = take_item(A, &slot, wid)) {
        estimate_body<SLOTS, false, true>(A, wid, item);
        __syncthreads();
    }
    estimate_body<SLOTS, false, true>(A, wid, kFlushTallies);
}

// The memory rule's out-of-line solve raises register use; its kernel still
// aims at four waves per SIMD (its recursion row shares LDS with the cut
// tables, so four blocks fit a CU) and spills the rest, which measured faster
// than three or two waves with fewer spills.
template <int SLOTS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void estimate_mem_kernel(EstimateArgs A)
{
    __shared__ int slot;
    const int wid = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    estimate_body<SLOTS, true>(A, wid, kZeroTallies);
    for (int item = take_item(A, &slot, wid); item >= 0; item = take_item(A, &slot, wid)) {
        estimate_body<SLOTS, true>(A, wid, item);
        __syncthreads();
    }
    estimate_body<SLOTS, true>(A, wid, kFlushTallies);
}

// ------------------------------------------------------------ interpolated communication latency

// Latency of v bytes in one profiled (volume, latency) table of K samples
// (vol[0] = 0, ascending): nothing moved costs nothing; otherwise linear
// between the samples around v, extended by the first or last segment.
__device__ __forceinline__ double tab_lat(const double* vol, const double* lat, int K, double v)
{
    if (!(v > 0.0)) return 0.0;
    int k = 1;
    while (k < K - 1 && v > vol[k]) ++k;
    return lat[k - 1] + (v - vol[k - 1]) * (lat[k] - lat[k - 1]) / (vol[k] - vol[k - 1]);
}

constexpr int kTabCacheBits = 8;
constexpr unsigned kTabCache = 1u << kTabCacheBits;   // bottleneck cache entries per block

struct TabBlockLds {
    float t[kLmax];
    float x[kLmax];
    float q[kLmax];
    double Pp[kLmax + 1];
    double Ap[kLmax + 1];
    double vol[2][kMaxTabPoints];     // link 0 inside a node, 1 across nodes
    double lat[2][kMaxTabPoints];
    double p_layer_max;               // largest parameter bytes of one layer
    double x_layer_min;               // smallest boundary activation bytes of one layer
    int32_t next_cell;
    int32_t share;                    // one kappa for all counts of the type: bottlenecks are shared
    double Upure[kLmax + kPad];       // prefix of the pure-compute per-sample cost (+inf padded)
    double Wpure[kLmax + 1];          // its bottleneck by degree (every degree up to the layer count)
    double head_p[kHeadLayers];       // parameter and activation bytes of the leading layers, as prefix
    double head_a[kHeadLayers];       //   differences (0 past the layer count)
    unsigned long long pure_cached[2];   // bit pp-1: the block's cache row of the pure split of pp is current
    WaveLds w[kWavesPerBlock];
    double cW[kTabCache];             // bottleneck cache of the (job, type): bottlenecks
    uint32_t ckey[kTabCache];         //   and their keys (0 empty)
};

// Bottleneck cache.  With one kappa for all counts of a type, a plan's
// per-microbatch layer costs depend on the cell only through (tp, b, whether
// dp tp > 1), so the bottleneck of pp stages over them is the same in every
// cell of the (job, type) that has a plan with that key: the first cell to
// solve it stores it, later cells price the degree without the recursion.
// Keys pack pp (8 bits), tp (5), the flag (1) and b (17 bits; larger batches
// do not share); bit 31 marks an entry whose value is still being written.
// Open addressing with linear probing; a full cache only stops sharing.
constexpr unsigned kTabBusy = 1u << 31;
constexpr int kTabProbe = 8;

__device__ __forceinline__ unsigned tab_key(int tp, bool flag, double b, int pp)
{
    return ((unsigned)b << 14) | ((flag ? 1u : 0u) << 13) | ((unsigned)tp << 8) | (unsigned)pp;
}

__device__ __forceinline__ unsigned tab_slot(unsigned key)
{
    return (key * 2654435761u) >> (32 - kTabCacheBits);
}

// Lane-parallel lookup: true and W when the bottleneck of `key` is cached.
__device__ __forceinline__ bool tab_cache_find(const TabBlockLds& B, unsigned key, double& W)
{
    unsigned h = tab_slot(key);
    for (int p = 0; p < kTabProbe; ++p) {
        const unsigned k = __hip_atomic_load(&B.ckey[h], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (k == key) {
            W = B.cW[h];
            return true;
        }
        if (k == 0u) return false;
        h = (h + 1u) & (kTabCache - 1u);
    }
    return false;
}

// One lane stores the bottleneck of `key` (nothing if the key is present or
// its probe window is full).
__device__ __forceinline__ void tab_cache_put(TabBlockLds& B, unsigned key, double W)
{
    unsigned h = tab_slot(key);
    for (int p = 0; p < kTabProbe; ++p) {
        const unsigned old = atomicCAS(&B.ckey[h], 0u, key | kTabBusy);
        if (old == 0u) {
            B.cW[h] = W;
            __hip_atomic_store(&B.ckey[h], key, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
            return;
        }
        if ((old & ~kTabBusy) == key) return;
        h = (h + 1u) & (kTabCache - 1u);
    }
}

// Per-microbatch cost of layers lane and lane+64 of plan (dp, tp) with b
// samples per microbatch (0 past L): compute, four tensor-parallel ring
// all-reduces of 2 (tp-1)/tp b x_l bytes on the intra-node link, the MoE
// all-to-all of b a2a_l bytes on the inter-node link; comm scaled by kappa.
__device__ __forceinline__ void tab_layer_costs(const TabBlockLds& B, int lane, const JobCtx& jb, const TypeDev& ty,
                                                int K, double kappa, int dp, int tp, double b, double (&c)[2])
{
    const double denom = (double)jb.Bg * ty.speed * (double)tp;
    const double ftp = 2.0 * (double)(tp - 1) / (double)tp;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int l = lane + 64 * s;
        c[s] = 0.0;
        if (l < jb.L) {
            double v = b * ((double)B.t[l] / denom);
            if (tp > 1) v += kappa * (4.0 * tab_lat(B.vol[0], B.lat[0], K, ftp * b * (double)B.x[l]));
            if (dp * tp > 1) v += kappa * tab_lat(B.vol[1], B.lat[1], K, b * (double)B.q[l]);
            c[s] = v;
        }
    }
}

// The plan's per-microbatch costs, prefix (into Wv.UD), bottleneck of pp
// stages (one-degree recursion) and canonical stages.
__device__ __forceinline__ Stages tab_partition(const TabBlockLds& B, WaveLds& Wv, int lane, const JobCtx& jb,
                                                const TypeDev& ty, int K, double kappa, int dp, int tp, int pp,
                                                double b, double& W)
{
    double c[2];
    tab_layer_costs(B, lane, jb, ty, K, kappa, dp, tp, b, c);
    seq_prefix<2, 2>(c[0], c[1], jb.L, lane, Wv.UD, Wv.UD + 1, true);
    Mask one;
    one.lo = pp <= 64 ? (1ull << (pp - 1)) : 0ull;
    one.hi = pp > 64 ? (1ull << (pp - 65)) : 0ull;
    W = 0.0;
    solve_dp(Wv, jb.L, one, lane, [&](int, double Wk, Mask mk) {
        W = Wk;
        return mk;
    });
    return canonical_stages<2>(Wv.UD, Wv.J, lane, jb.L, pp, W);
}

// Iteration time of plan (dp, tp, pp, m) on stages sg under the tables
// (+inf if a stage does not fit):
//   T = sum_k (W_k + p2p_k) + (m-1) max_k W_k + max_k AR_k,
//   W_k the stage's per-microbatch cost, p2p_k = kappa 2 f_pp(b x_last)
//   (k < pp-1), AR_k = kappa f_dp(2 (dp-1)/dp P_k/tp) (dp > 1), memory as in
//   the balanced model.
__device__ __forceinline__ double tab_price(const TabBlockLds& B, WaveLds& Wv, int lane, const JobCtx& jb,
                                            const TypeDev& ty, int K, const Cell& cell, int dp, int tp, int pp,
                                            int m, double b, const Stages& sg)
{
    const int lpp = cell.n <= ty.gpn ? 0 : 1;
    const int grp = dp * tp;
    const int ldp = tiles_node(ty, grp) ? 0 : 1;
    const double fdp = 2.0 * (double)(dp - 1) / (double)dp;
    double fill = 0.0, wmax = 0.0, armax = 0.0, memmax = 0.0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int k = lane + 64 * h;
        if (k < pp) {
            const int lo = h == 0 ? sg.lo0 : sg.lo1;
            const int hi = h == 0 ? sg.hi0 : sg.hi1;
            const double Wk = Wv.UD[2 * hi] - Wv.UD[2 * lo];
            const double Pk = B.Pp[hi] - B.Pp[lo];
            const double Ak = B.Ap[hi] - B.Ap[lo];
            double p2p = 0.0;
            if (k < pp - 1) p2p = cell.kappa * (2.0 * tab_lat(B.vol[lpp], B.lat[lpp], K, b * (double)B.x[hi - 1]));
            double AR = 0.0;
            if (dp > 1) AR = cell.kappa * tab_lat(B.vol[ldp], B.lat[ldp], K, fdp * (Pk / (double)tp));
            const int inflight = m < pp - k ? m : pp - k;
            const double Mem = 4.0 * Pk / (double)tp + (double)inflight * b * Ak / (double)tp;
            fill += Wk + p2p;
            wmax = fmax(wmax, Wk);
            armax = fmax(armax, AR);
            memmax = fmax(memmax, Mem);
        }
    }
    double rs[1] = {fill};
    double rm[3] = {wmax, armax, memmax};
    wave_reduce<OpSum, 1>(rs);
    wave_reduce<OpMax, 3>(rm);
    if (!(rm[2] <= ty.mem)) return kInf;
    return rs[0] + (double)(m - 1) * rm[0] + rm[1];
}

// Lower bound of the time of plan (dp, tp, pp, m) over every split, or +inf
// when no split can fit memory, from its per-microbatch costs alone: the
// stages tile the layers (W_max >= sum c / pp and >= max c), each of the pp-1
// boundaries moves at least the smallest boundary activation, the largest
// stage holds at least max(P / pp, max p_l) of parameters, and f is
// non-decreasing.  A relative margin of 1e-9 covers the sums' rounding.
// The sum and the largest of the per-microbatch costs depend on the plan only
// through (tp, b, dp tp > 1): the wave keeps those of the cell's current tp in
// a small table in its UD row (unused until the plans are priced): keys at
// [0, 64) (b, negated when dp tp = 1), sums at [64, 128), largest at [128, 192);
// `nc` entries (uniform).
__device__ __forceinline__ double tab_bound(const TabBlockLds& B, WaveLds& Wv, int lane, const JobCtx& jb,
                                            const TypeDev& ty, int K, const Cell& cell, int dp, int tp, int pp,
                                            int m, double b, int& nc)
{
    const double plb = fmax(B.Pp[jb.L] / (double)pp, B.p_layer_max);
    if (4.0 * plb > ty.mem * (double)tp * (1.0 + 1e-9)) return kInf;
    // the stage holding layer l (l <= kHeadLayers) has at most l - 1 stages
    // before it: at least min(m, pp - l + 1) microbatches in flight, and that
    // layer's own bytes lower-bound its memory term by term
#pragma unroll
    for (int l = 1; l <= kHeadLayers; ++l) {
        const int r = pp - l + 1;
        const int f = m < r ? m : (r > 1 ? r : 1);
        const double memb = 4.0 * B.head_p[l - 1] / (double)tp + (double)f * b * B.head_a[l - 1] / (double)tp;
        if (!(memb <= ty.mem)) return kInf;
    }
    const double key = dp * tp > 1 ? b : -b;
    const unsigned long long hit = __ballot(lane < nc && Wv.UD[lane] == key);
    double UL, cmax;
    if (hit) {
        const int e = __builtin_amdgcn_readfirstlane((int)__builtin_ctzll(hit));
        UL = Wv.UD[64 + e];
        cmax = Wv.UD[128 + e];
    } else {
        double c[2];
        tab_layer_costs(B, lane, jb, ty, K, cell.kappa, dp, tp, b, c);
        double rs[1] = {c[0] + c[1]};
        double rm[1] = {fmax(c[0], c[1])};
        wave_reduce<OpSum, 1>(rs);
        wave_reduce<OpMax, 1>(rm);
        UL = rs[0];
        cmax = rm[0];
        tally(Wv, lane, kAlgOps, 4ull * (unsigned)jb.L);
        if (nc < 64) {
            if (lane == 0) {
                Wv.UD[nc] = key;
                Wv.UD[64 + nc] = UL;
                Wv.UD[128 + nc] = cmax;
            }
            wave_sync();
            ++nc;
        }
    }
    const double Wlb = fmax(UL / (double)pp, cmax);
    const int lpp = cell.n <= ty.gpn ? 0 : 1;
    const int grp = dp * tp;
    const int ldp = tiles_node(ty, grp) ? 0 : 1;
    const double p2p = pp > 1 ? cell.kappa * (2.0 * tab_lat(B.vol[lpp], B.lat[lpp], K, b * B.x_layer_min)) : 0.0;
    const double ar = dp > 1
        ? cell.kappa * tab_lat(B.vol[ldp], B.lat[ldp], K, 2.0 * (double)(dp - 1) / (double)dp * (plb / (double)tp))
        : 0.0;
    return (UL + (double)(pp - 1) * p2p + (double)(m - 1) * Wlb + ar) * (1.0 - 1e-9);
}

// Plan-buffer key of the interpolated-tables kernel: pp << 12 | tp << 7 | m,
// with the top bit set once the plan is priced.
constexpr unsigned kTabPriced = 1u << 31;
constexpr unsigned kTabKeyMask = kTabPriced - 1u;

// Every cell under interpolated communication latency: a block works on one
// (job, type) at a time (taken from the queue), its waves taking counts.  Every plan of a cell has the balanced
// partition of its own per-microbatch costs.  Those costs depend on the plan
// only through tp, b and whether dp tp > 1, and for fixed tp and b each
// pipeline degree fixes dp and hence m, so the plans of a cell sharing (tp, b,
// dp tp > 1) form a group that differs only in pp: one recursion up to the
// group's largest degree gives every member's bottleneck, and each member is
// priced as soon as its row is done.  With bound pruning, the plans' lower
// bounds come first, then the unpriced plan of least bound is priced with its
// group, again and again, until every bound left lies past the tie window of
// the best time priced so far (those plans can neither be the best nor tie
// with it): a group takes only members within the window and drops the
// degrees the window excludes as it tightens.  Then the cell's choice as in
// estimate_kernel.
__device__ __forceinline__ void estimate_tab_body(const EstimateArgs& A, int wid, int item)
{
    __shared__ TabBlockLds B;
    // lane index counted per item and per cell (as in estimate_body)
    int lane0;
    __asm__ volatile("" : "=v"(lane0) : "0"((int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u))));
    const int lane = lane0;
    const int tid = wid * 64 + lane;
    WaveLds& Wv = B.w[wid];
    if (item < 0) {
        block_tallies(A, Wv, lane, item);
        return;
    }
    uint8_t* const pcache = A.pure_cuts + (size_t)blockIdx.x * kPureCutBytes;

    const int j = item / A.n_types;
    const int g = item - j * A.n_types;
    const int off = A.layer_offset[j];
    JobCtx jb;
    jb.L = A.layer_offset[j + 1] - off;
    jb.Bg = A.batch[j];
    jb.moe = false;
    const TypeDev ty = A.types[g];
    const int K = A.tab_k;

    if (tid < jb.L) {
        B.t[tid] = A.t[off + tid];
        B.x[tid] = A.x[off + tid];
        B.q[tid] = A.q[off + tid];
    }
    if (tid < 2 * K) {
        const int link = tid / K, k = tid - link * K;
        const long long base = ((long long)g * 2 + link) * K + k;
        B.vol[link][k] = A.tab_vol[base];
        B.lat[link][k] = A.tab_lat[base];
    }
    if (wid == 0 || wid == 1) {
        const float* src = (wid == 0 ? A.p : A.a) + off;
        const double v0 = lane < jb.L ? (double)src[lane] : 0.0;
        const double v1 = lane + 64 < jb.L ? (double)src[lane + 64] : 0.0;
        seq_prefix<1, 2>(v0, v1, jb.L, lane, wid == 0 ? B.Pp : B.Ap, Wv.UD + 1, false);
        if (lane < kHeadLayers) {
            const double* pre = wid == 0 ? B.Pp : B.Ap;
            (wid == 0 ? B.head_p : B.head_a)[lane] = lane < jb.L ? pre[lane + 1] - pre[lane] : 0.0;
        }
        if (wid == 0) {
            const double pm = wave_reduce1<OpMax>(fmax(v0, v1));
            if (lane == 0) B.p_layer_max = pm;
        }
    } else if (wid == 2) {
        const double x0 = lane < jb.L ? (double)A.x[off + lane] : kInf;
        const double x1 = lane + 64 < jb.L ? (double)A.x[off + lane + 64] : kInf;
        const double xm = wave_reduce1<OpMin>(fmin(x0, x1));
        if (lane == 0) B.x_layer_min = xm;
        // the pure-compute problem for every degree: its canonical splits are
        // the first candidates of the groups' bottleneck certificates
        build_prefix_u<1>(A.t + off, A.x + off, A.q + off, B.Upure, Wv.UD + 1, lane, jb, ty, 1.0, 1, false);
        for (int e = lane; e < kLmax + kPad; e += 64) Wv.UD[2 * e] = B.Upure[e];
        wave_sync();
        solve_dp(Wv, jb.L, ballot_mask(1 + lane <= jb.L, 65 + lane <= jb.L), lane, [&](int pp, double W, Mask m) {
            if (lane == 0) B.Wpure[pp] = W;
            return m;
        });
        tally(Wv, lane, kProblems, 1);
        tally(Wv, lane, kAlgOps, 8ull * (unsigned)jb.L);
    } else {
        bool same = true;
        for (int c = lane; c < A.n_counts; c += 64) same &= A.kappa[g * A.n_counts + c] == A.kappa[g * A.n_counts];
        const bool uni = __ballot(!same) == 0ull;
        for (int h = lane; h < (int)kTabCache; h += 64) B.ckey[h] = 0u;
        if (lane == 0) {
            B.share = (uni && A.n_counts > 1 && jb.Bg < (1 << 17)) ? 1 : 0;
            B.pure_cached[0] = 0ull;
            B.pure_cached[1] = 0ull;
        }
    }
    if (tid == 0) B.next_cell = 0;
    if (wid == 0) tally(Wv, lane, kCells, (unsigned long long)A.n_counts);
    __syncthreads();
    const bool share = B.share != 0;

    for (;;) {
        int lane;
        __asm__ volatile("" : "=v"(lane) : "0"((int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u))));
        int cix = 0;
        if (lane == 0) cix = atomicAdd(&B.next_cell, 1);
        cix = __builtin_amdgcn_readfirstlane(cix);
        if (cix >= A.n_counts) break;
        const int ci = A.count_order[cix];
        Cell cell;
        cell.n = A.counts[ci];
        cell.kappa = (double)A.kappa[g * A.n_counts + ci];
        cell.B_pp = 0.0;
        cell.c_p2p = 0.0;
        // the plans: keys and lower bounds
        int np = 0, nskip = 0;
        for (int tp = 1; tp <= cell.n && tp <= ty.gpn; ++tp) {
            if (!tiles_node(ty, tp) || exact_quot(cell.n, tp) * tp != cell.n) continue;
            const int qn = exact_quot(cell.n, tp);
            int nc = 0;                     // the bounds' cost sums of this tp
            for (int pp = 1; pp <= qn && pp <= jb.L; ++pp) {
                const int dp = exact_quot(qn, pp);
                if (dp * pp != qn) continue;
                for (int mi = 0; mi < A.n_m; ++mi) {
                    const int m = A.m_values[mi];
                    const double dm = (double)(dp * m);
                    const double bq = rint((double)jb.Bg * rcp_approx(dm));   // exact when dm divides Bg
                    if (!(bq * dm == (double)jb.Bg)) continue;
                    const double lb = A.prune ? tab_bound(B, Wv, lane, jb, ty, K, cell, dp, tp, pp, m, bq, nc) : 0.0;
                    if (lane == 0 && np < kMaxPlans) {
                        Wv.planT[np] = lb;
                        Wv.planKey[np] = ((unsigned)pp << 12) | ((unsigned)tp << 7) | (unsigned)m;
                    }
                    ++np;
                }
            }
        }
        if (np > kMaxPlans) {
            tally(Wv, lane, kOverflow, 1);
            np = kMaxPlans;
        }
        wave_sync();
        // price plan e0 of the buffer and the unpriced plans of its group (each
        // slot receives its time and the priced flag); returns the best time
        // so far.  Wv.lbnd[d - 1] holds the member of degree d (-1: none).
        auto price_group = [&](int e0, double best_in) -> double {
            const unsigned key0 = Wv.planKey[e0] & kTabKeyMask;
            const int pp0 = (int)(key0 >> 12);
            const int tp0 = (int)((key0 >> 7) & 0x1Fu);
            const int dp0 = exact_quot(cell.n, tp0 * pp0);
            const double bq0 = rint((double)jb.Bg / (double)(dp0 * (int)(key0 & 0x7Fu)));
            const bool fl0 = dp0 * tp0 > 1;
            const double lim0 = best_in * (1.0 + A.tie_eps);
            Wv.lbnd[lane] = -1.0;
            Wv.lbnd[lane + 64] = -1.0;
            wave_sync();
            for (int e = lane; e < np; e += 64) {
                const unsigned k = Wv.planKey[e];
                if (k & kTabPriced) continue;
                const int pp = (int)(k >> 12);
                const int tp = (int)((k >> 7) & 0x1Fu);
                if (tp != tp0) continue;
                const int dp = exact_quot(cell.n, tp * pp);
                if ((dp * tp > 1) != fl0 || rint((double)jb.Bg / (double)(dp * (int)(k & 0x7Fu))) != bq0) continue;
                const double lbe = Wv.planT[e];
                if (e != e0 && A.prune && !(lbe < kInf && lbe <= lim0)) continue;
                Wv.lbnd[pp - 1] = (double)e;      // degrees of a group are distinct
            }
            wave_sync();
            const Mask tm = ballot_mask(Wv.lbnd[lane] >= 0.0, Wv.lbnd[lane + 64] >= 0.0);
            double c[2];
            tab_layer_costs(B, lane, jb, ty, K, cell.kappa, dp0, tp0, bq0, c);
            seq_prefix<2, 2>(c[0], c[1], jb.L, lane, Wv.UD, Wv.UD + 1, true);
            tally(Wv, lane, kAlgOps, 8ull * (unsigned)jb.L);
            double bst = best_in;
            // prices degree pp of the group at bottleneck W; returns the degrees still wanted
            auto price_deg = [&](int pp, double W, Mask mk) -> Mask {
                const int e = (int)Wv.lbnd[pp - 1];
                const int dp = exact_quot(cell.n, tp0 * pp);
                const int m = (int)(Wv.planKey[e] & 0x7Fu);
                const Stages sg = canonical_stages<2>(Wv.UD, Wv.J, lane, jb.L, pp, W);
                const double T = tab_price(B, Wv, lane, jb, ty, K, cell, dp, tp0, pp, m, bq0, sg);
                tally(Wv, lane, kAlgOps, 4ull * (unsigned)jb.L + 12ull * (unsigned)pp + 40ull);
                wave_sync();
                if (lane == 0) {
                    Wv.planT[e] = T;
                    Wv.planKey[e] |= kTabPriced;
                }
                wave_sync();
                bst = fmin(bst, T);
                Mask rest = mk;                      // degrees still to come
                if (pp <= 64) rest.lo &= ~(1ull << (pp - 1)); else rest.hi &= ~(1ull << (pp - 65));
                if (!A.prune) return rest;
                // members whose bound now lies past the window are left to the
                // main loop, which skips them
                const double lim = bst * (1.0 + A.tie_eps);
                const int ea = (int)Wv.lbnd[lane], eb = (int)Wv.lbnd[lane + 64];
                const bool ka = ea >= 0 && Wv.planT[ea] <= lim;
                const bool kb = eb >= 0 && Wv.planT[eb] <= lim;
                return rest & ballot_mask(ka, kb);
            };
            // degrees another cell of this (job, type) has solved are priced
            // first, from the cache; the recursion runs for the others only
            Mask want = tm, hit{0ull, 0ull};
            if (share) {
                double w0 = 0.0, w1 = 0.0;
                const bool h0 = ((tm.lo >> lane) & 1ull) && tab_cache_find(B, tab_key(tp0, fl0, bq0, 1 + lane), w0);
                const bool h1 = ((tm.hi >> lane) & 1ull) && tab_cache_find(B, tab_key(tp0, fl0, bq0, 65 + lane), w1);
                hit = ballot_mask(h0, h1);
                for (int pp = hit.next(1); pp; pp = hit.next(pp + 1))
                    if (want.test(pp)) want = price_deg(pp, pp <= 64 ? bcast(w0, pp - 1) : bcast(w1, pp - 65), want);
            }
            Mask todo{want.lo & ~hit.lo, want.hi & ~hit.hi};
            // the largest degrees left first: a certified bottleneck spares the
            // recursion their rows
            for (int pc = todo.last(); pc >= kCertMinDegree; pc = todo.last()) {
                const double wc = certified_bottleneck(
                    pure_split(B.Upure, B.Wpure[pc], B.pure_cached, Wv, pcache, lane, jb.L, pc), Wv, lane, jb.L, pc);
                if (!(wc >= 0.0)) break;
                if (share && lane == 0) tab_cache_put(B, tab_key(tp0, fl0, bq0, pc), wc);
                todo = price_deg(pc, wc, todo);
            }
            if (todo.any()) {
                tally(Wv, lane, kProblems, 1);
                solve_dp(Wv, jb.L, todo, lane, [&](int pp, double W, Mask mk) {
                    if (share && lane == 0) tab_cache_put(B, tab_key(tp0, fl0, bq0, pp), W);
                    return price_deg(pp, W, mk);
                });
            }
            return bst;
        };
        if (A.prune) {
            // best first: the unpriced plan of least bound (and its group),
            // until every bound left lies past the tie window of the best time
            double best = kInf;
            for (;;) {
                double bl = kInf;
                for (int e = lane; e < np; e += 64)
                    if (!(Wv.planKey[e] & kTabPriced)) bl = fmin(bl, Wv.planT[e]);
                const double bmin = wave_reduce1<OpMin>(bl);
                if (!(bmin < kInf && bmin <= best * (1.0 + A.tie_eps))) break;
                double il = -1.0;
                for (int e = lane; e < np; e += 64)
                    if (!(Wv.planKey[e] & kTabPriced) && Wv.planT[e] == bmin) il = (double)e;
                best = price_group((int)wave_reduce1<OpMax>(il), best);
            }
            // the rest can neither be the best nor tie with it
            double ns = 0.0;
            for (int e = lane; e < np; e += 64)
                if (!(Wv.planKey[e] & kTabPriced)) {
                    Wv.planT[e] = kInf;
                    ns += 1.0;
                }
            nskip = (int)wave_reduce1<OpSum>(ns);
            wave_sync();
        } else {
            for (int e = 0; e < np; ++e)
                if (!(Wv.planKey[e] & kTabPriced)) price_group(e, kInf);
        }
        wave_sync();

        double tl = kInf;
        for (int e = lane; e < np; e += 64) tl = fmin(tl, Wv.planT[e]);
        const double tmin = wave_reduce1<OpMin>(tl);
        const long long cidx = ((long long)j * A.n_types + g) * A.n_counts + ci;
        tally(Wv, lane, kPlans, (unsigned long long)(np - nskip));
        if (!(tmin < kInf)) {
            tally(Wv, lane, kInfeasible, 1);
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
        const double tlim = tmin * (1.0 + A.tie_eps);
        // the smallest key within the window and its entry in one reduction
        double kl = kInf;
        for (int e = lane; e < np; e += 64)
            if (Wv.planT[e] <= tlim) kl = fmin(kl, (double)(Wv.planKey[e] & kTabKeyMask) * 256.0 + (double)e);
        const double kv = wave_reduce1<OpMin>(kl);
        const unsigned kbest = (unsigned)(kv * (1.0 / 256.0));
        int ib = (int)(kv - (double)kbest * 256.0);
        ib = ib < 0 ? 0 : (ib >= np ? np - 1 : ib);
        const double Tb = Wv.planT[ib];
        const int pp = (int)(kbest >> 12);
        const int tp = (int)((kbest >> 7) & 0x1Fu);
        const int m = (int)(kbest & 0x7Fu);
        const int dp = exact_quot(cell.n, tp * pp);
        if (lane == 0) {
            A.t_iter[cidx] = (float)Tb;
            A.thr[cidx] = (float)((double)jb.Bg / Tb);
            A.plan[cidx] = (unsigned)dp | ((unsigned)tp << 11) | ((unsigned)pp << 16) | ((unsigned)m << 24) |
                           (1u << 31);
        }
        if (A.cuts) {
            // re-derive the winner's stages (the recursion's entries are not tallied twice)
            const unsigned long long e0 = Wv.tally[kDpEntries];
            const double bw = rint((double)jb.Bg / (double)(dp * m));
            double W;
            const Stages sg = tab_partition(B, Wv, lane, jb, ty, K, cell.kappa, dp, tp, pp, bw, W);
            if (lane == 0) Wv.tally[kDpEntries] = e0;
            uint8_t* row = A.cuts + cidx * A.cuts_stride;
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const int idx = lane + 64 * s;
                const int en = s == 0 ? +sg.hi0 : +sg.hi1;
                if (idx < A.cuts_stride) row[idx] = (idx < pp - 1) ? (uint8_t)en : (uint8_t)0xFF;
            }
            for (int e = 128 + lane; e < A.cuts_stride; e += 64) row[e] = 0xFF;
        }
        wave_sync();
    }

}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void estimate_tab_kernel(EstimateArgs A)
{
    __shared__ int slot;
    const int wid = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    estimate_tab_body(A, wid, kZeroTallies);
    for (int item = take_item(A, &slot, wid); item >= 0; item = take_item(A, &slot, wid)) {
        estimate_tab_body(A, wid, item);
        __syncthreads();
    }
    estimate_tab_body(A, wid, kFlushTallies);
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

// The no-allocation estimate's scratch: library-owned tables, work order and
// counters of one call, on every device the library runs on, held until the
// process ends.  Host code never passes this name to a kernel (on the host it
// only stands for the symbol); it uses the address scratch_address returns.
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

hipError_t scratch_address(int device, void** out)
{
    static std::mutex mu;
    static void* addr[kMaxScratchDevices] = {};
    if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[device] = p;
    }
    *out = addr[device];
    return hipSuccess;
}

hipError_t launch_estimate(const EstimateArgs& args, hipStream_t stream)
{
    if (args.n_items <= 0 || args.n_blocks <= 0) return hipSuccess;
    const dim3 grid((unsigned)args.n_blocks), block(256);
    if (args.tab_k > 0) {
        hipLaunchKernelGGL(estimate_tab_kernel, grid, block, 0, stream, args);
    } else if (args.exact_t) {
        if (args.share_tp)
            hipLaunchKernelGGL((estimate_ext_kernel<kSlotsShared>), grid, block, 0, stream, args);
        else
            hipLaunchKernelGGL((estimate_ext_kernel<1>), grid, block, 0, stream, args);
    } else if (args.mem_rule) {
        if (args.share_tp)
            hipLaunchKernelGGL((estimate_mem_kernel<kSlotsShared>), grid, block, 0, stream, args);
        else
            hipLaunchKernelGGL((estimate_mem_kernel<1>), grid, block, 0, stream, args);
    } else {
        if (args.share_tp)
            hipLaunchKernelGGL((estimate_kernel<kSlotsShared>), grid, block, 0, stream, args);
        else
            hipLaunchKernelGGL((estimate_kernel<1>), grid, block, 0, stream, args);
    }
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
