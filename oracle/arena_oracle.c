/*
 * CPU oracle for the plan-space estimator: TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke entry and the benchmark's CPU-baseline leg
 * may load this library.  The product path never calls it; it shares no
 * code, header or constant with the HIP library.
 *
 * It computes, plainly and slowly, in IEEE double precision from the f32
 * input tables, what the estimator computes for one (job, GPU type, GPU
 * count) cell:
 *   - every adaptive-parallelism plan (dp, tp, pp, m) of the cell
 *     (the joint space of Eq. 1 restricted to one scheduling plan; the grid
 *      sharding of Sec. 3.2 fixes resources and pipeline degree);
 *   - for each plan, the contiguous stage partition with the smallest
 *     slowest-stage time (the balanced-stage criterion of Sec. 3.2: a
 *     pipeline is bottlenecked by its slowest stage), found by the textbook
 *     recursion over prefixes, and the canonical (lexicographically smallest)
 *     optimal cut vector; under the memory-constrained rule the same
 *     criterion restricted to the cut vectors whose every stage fits the
 *     GPU's memory (Sec. 3.3 chooses within memory limits);
 *   - the plan's iteration time: the 1F1B model of Sec. 3.4 (first
 *     microbatch through every stage, plus B-1 further microbatches on the
 *     slowest stage with point-to-point overlapped), stage latency as the sum
 *     of its operators (Sec. 3.4), intra-stage communication in the stage
 *     (Eq. 4's per-microbatch term), gradient all-reduce once per iteration
 *     (Eq. 4's once-per-iteration term), latency proportional to volume
 *     (Sec. 3.4), memory limits (Sec. 3.3);
 *   - the best plan of the cell, its iteration time T and throughput
 *     Bg / T: one entry of the throughput matrix of Eq. 5;
 *   - optionally (the *_tab entries) communication latency interpolated in
 *     per-link tables of profiled (volume, latency) samples (Sec. 3.4)
 *     instead of volume / bandwidth.
 *
 * Readings where the paper leaves the model open (units, memory model,
 * link choice, tie-breaks) are listed in the repository's design notes;
 * each function below states which one it follows.
 *
 * Parity pins: W* is pinned against brute force over every cut vector,
 * the cuts against the brute-force lexicographic minimum, the plan price
 * against hand-derived cells, closed forms and invariants (see tests/).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <stdio.h>

#define ORACLE_MAX_L 128

/* Allocation that cannot fail silently: a test oracle that ran out of memory
 * must stop rather than return a partial answer. */
static void* xrealloc(void* old, size_t bytes)
{
    void* p = realloc(old, bytes ? bytes : 1);
    if (!p) {
        fprintf(stderr, "arena oracle: out of memory (%zu bytes)\n", bytes);
        abort();
    }
    return p;
}

/* ------------------------------------------------------------------ */
/* Stage partition                                                     */
/* ------------------------------------------------------------------ */

/* U[0] = 0, U[i] = U[i-1] + u[i-1]: left to right. */
void oracle_prefix(const double* u, int L, double* U)
{
    U[0] = 0.0;
    for (int i = 1; i <= L; ++i) U[i] = U[i - 1] + u[i - 1];
}

/* Segment [lo, hi) of the prefix U. */
static double seg(const double* U, int lo, int hi) { return U[hi] - U[lo]; }

/* Brute force over every cut vector 0 < c_1 < ... < c_{pp-1} < L, visited in
 * lexicographic order; returns min over vectors of the largest segment and
 * writes the first (lexicographically smallest) vector that attains it.
 * This is the definition of the balanced partition (Sec. 3.2), written out.
 * Cost C(L-1, pp-1): for small L only. */
typedef struct {
    const double* U;
    int L, pp;
    int cur[ORACLE_MAX_L + 1];
    int best[ORACLE_MAX_L + 1];
    double best_w;
} bf_state;

static void bf_rec(bf_state* s, int k, int start, double run_max)
{
    /* k = index of the cut being placed (1..pp-1); cur[k-1] is fixed. */
    if (k == s->pp) {
        double w = seg(s->U, s->cur[k - 1], s->L);
        double m = run_max > w ? run_max : w;
        if (m < s->best_w) {
            s->best_w = m;
            memcpy(s->best, s->cur, sizeof(int) * (size_t)(s->pp + 1));
        }
        return;
    }
    /* c_k ranges so that pp-k more non-empty segments still fit. */
    for (int c = start; c <= s->L - (s->pp - k); ++c) {
        double w = seg(s->U, s->cur[k - 1], c);
        double m = run_max > w ? run_max : w;
        s->cur[k] = c;
        bf_rec(s, k + 1, c + 1, m);
    }
}

double oracle_bottleneck_bruteforce(const double* U, int L, int pp, int* cuts)
{
    if (L < 1 || pp < 1 || pp > L || L > ORACLE_MAX_L) return NAN;
    bf_state s;
    s.U = U; s.L = L; s.pp = pp; s.best_w = INFINITY;
    s.cur[0] = 0;
    bf_rec(&s, 1, 1, -INFINITY);
    if (cuts)
        for (int k = 1; k < pp; ++k) cuts[k - 1] = s.best[k];
    return s.best_w;
}

/* Textbook recursion: D_1(i) = U_i - U_0,
 * D_k(i) = min over j in [k-1, i-1] of max(D_{k-1}(j), U_i - U_j);
 * W*(pp) = D_pp(L).  O(pp L^2). */
double oracle_bottleneck_dp(const double* U, int L, int pp)
{
    if (L < 1 || pp < 1 || pp > L || L > ORACLE_MAX_L) return NAN;
    double prev[ORACLE_MAX_L + 1], cur[ORACLE_MAX_L + 1];
    for (int i = 0; i <= L; ++i) prev[i] = INFINITY;
    for (int i = 1; i <= L; ++i) prev[i] = seg(U, 0, i);
    for (int k = 2; k <= pp; ++k) {
        for (int i = 0; i <= L; ++i) cur[i] = INFINITY;
        for (int i = k; i <= L; ++i) {
            double best = INFINITY;
            for (int j = k - 1; j <= i - 1; ++j) {
                double a = prev[j], b = seg(U, j, i);
                double m = a > b ? a : b;
                if (m < best) best = m;
            }
            cur[i] = best;
        }
        memcpy(prev, cur, sizeof(cur));
    }
    return prev[L];
}

/* Canonical cuts: c_pp = L and, right to left,
 * c_k = smallest c >= k with U_{c_{k+1}} - U_c <= W.
 * This is the lexicographically smallest cut vector whose segments are all
 * <= W (front stages as short as possible). */
void oracle_canonical_cuts(const double* U, int L, int pp, double W, int* cuts)
{
    int next = L;
    for (int k = pp - 1; k >= 1; --k) {
        int c = k;
        while (c < next - 1 && seg(U, c, next) > W) ++c;
        cuts[k - 1] = c;
        next = c;
    }
}

/* ------------------------------------------------------------------ */
/* Memory-constrained stage partition                                  */
/* ------------------------------------------------------------------ */

/* One plan's memory model seen from the partition: stage k (0-based) of a
 * pp-stage 1F1B pipeline over layers [lo, hi) needs
 *   4 P/tp + min(m, pp-k) b A/tp  bytes,
 * P and A the parameter and activation bytes of its layers (summed left to
 * right in double), and fits when that is at most mem. */
typedef struct {
    const double* p;   /* per-layer parameter bytes */
    const double* a;   /* per-layer activation bytes per sample */
    int L, m, tp;
    double b, mem;
} omem;

static int fits_sums(const omem* M, double P, double A, int k, int pp)
{
    int inflight = M->m < pp - k ? M->m : pp - k;
    double Mem = 4.0 * P / (double)M->tp + (double)inflight * M->b * A / (double)M->tp;
    return Mem <= M->mem;
}

static int stage_fits(const omem* M, int lo, int hi, int k, int pp)
{
    double P = 0.0, A = 0.0;
    for (int l = lo; l < hi; ++l) { P += M->p[l]; A += M->a[l]; }
    return fits_sums(M, P, A, k, pp);
}

/* Brute force: every cut vector in lexicographic order; among those whose
 * every stage fits, the least largest segment and the first vector attaining
 * it.  +inf (cuts untouched) when no vector fits.  Small L only. */
typedef struct {
    const double* U;
    const omem* M;
    int L, pp;
    int cur[ORACLE_MAX_L + 1];
    int best[ORACLE_MAX_L + 1];
    double best_w;
} bfm_state;

static void bfm_rec(bfm_state* s, int k, double run_max)
{
    /* stages 0..k-2 are placed and fit; cur[k-1] starts stage k-1 */
    if (k == s->pp) {
        if (!stage_fits(s->M, s->cur[k - 1], s->L, k - 1, s->pp)) return;
        double w = seg(s->U, s->cur[k - 1], s->L);
        double m = run_max > w ? run_max : w;
        if (m < s->best_w) {
            s->best_w = m;
            memcpy(s->best, s->cur, sizeof(int) * (size_t)(s->pp + 1));
        }
        return;
    }
    for (int c = s->cur[k - 1] + 1; c <= s->L - (s->pp - k); ++c) {
        if (!stage_fits(s->M, s->cur[k - 1], c, k - 1, s->pp)) continue;
        double w = seg(s->U, s->cur[k - 1], c);
        double m = run_max > w ? run_max : w;
        s->cur[k] = c;
        bfm_rec(s, k + 1, m);
    }
}

static double bottleneck_mem_bruteforce(const double* U, const omem* M, int pp, int* cuts)
{
    bfm_state s;
    s.U = U; s.M = M; s.L = M->L; s.pp = pp; s.best_w = INFINITY;
    s.cur[0] = 0;
    bfm_rec(&s, 1, -INFINITY);
    if (cuts && s.best_w < INFINITY)
        for (int k = 1; k < pp; ++k) cuts[k - 1] = s.best[k];
    return s.best_w;
}

/* Recursion over suffixes, stages counted from the back (a stage's number of
 * in-flight microbatches, min(m, pp-k), depends only on how many stages
 * follow it, so suffix problems do not depend on pp):
 *   G_0(L) = -inf, G_0(i) = +inf for i < L;
 *   G_t(i) = min over e in (i, L] with layers [i, e) fitting as the t-th
 *            stage from the back of max(U_e - U_i, G_{t-1}(e)).
 * G_t(i) is the least largest segment over the splits of [i, L) into t
 * non-empty stages that all fit.  G has (pp+1)(L+1) entries.  O(pp L^2): the
 * memory sums of [i, e) grow with e one layer at a time (the same left-to-
 * right sums as stage_fits). */
static void mem_recursion(const double* U, const omem* M, int pp, double* G)
{
    int L = M->L, L1 = L + 1;
    for (int i = 0; i <= L; ++i) G[i] = (i == L) ? -INFINITY : INFINITY;
    for (int t = 1; t <= pp; ++t) {
        for (int i = 0; i <= L; ++i) {
            double best = INFINITY, P = 0.0, A = 0.0;
            for (int e = i + 1; e <= L; ++e) {
                P += M->p[e - 1];
                A += M->a[e - 1];
                /* as the t-th stage from the back it is stage pp - t */
                if (!fits_sums(M, P, A, pp - t, pp)) continue;
                double g = G[(t - 1) * L1 + e], w = seg(U, i, e);
                double v = w > g ? w : g;
                if (v < best) best = v;
            }
            G[t * L1 + i] = best;
        }
    }
}

/* W*_mem(pp) = G_pp(0) and the lexicographically smallest cut vector that
 * attains it with every stage fitting: each cut, left to right, is the
 * smallest position such that the stage it closes fits, is at most W, and
 * the rest of the layers still split into the remaining stages within W.
 * +inf (cuts untouched) when no split fits. */
static double bottleneck_mem(const double* U, const omem* M, int pp, int* cuts)
{
    int L = M->L, L1 = L + 1;
    double* G = (double*)xrealloc(NULL, sizeof(double) * (size_t)(pp + 1) * (size_t)L1);
    mem_recursion(U, M, pp, G);
    double W = G[pp * L1 + 0];
    if (cuts && W < INFINITY) {
        int prev = 0;
        for (int k = 1; k < pp; ++k) {
            int c = prev + 1;
            while (!(seg(U, prev, c) <= W && stage_fits(M, prev, c, k - 1, pp) &&
                     G[(pp - k) * L1 + c] <= W))
                ++c;
            cuts[k - 1] = c;
            prev = c;
        }
    }
    free(G);
    return W;
}

/* Exposed for tests: p, a per-layer bytes, b samples per microbatch.
 * Returns W (+inf if no split fits); cuts receives pp - 1 cuts. */
double oracle_bottleneck_mem(const double* U, const double* p, const double* a, int L, int pp,
                             int m, double b, int tp, double mem, int brute, int* cuts)
{
    if (L < 1 || pp < 1 || pp > L || L > ORACLE_MAX_L || m < 1 || tp < 1) return NAN;
    omem M;
    M.p = p; M.a = a; M.L = L; M.m = m; M.tp = tp; M.b = b; M.mem = mem;
    return brute ? bottleneck_mem_bruteforce(U, &M, pp, cuts) : bottleneck_mem(U, &M, pp, cuts);
}

/* ------------------------------------------------------------------ */
/* Plan pricing                                                        */
/* ------------------------------------------------------------------ */

typedef struct {
    int L, Bg;
    const float *t, *p, *a, *x, *a2a;
} ojob;

typedef struct {
    double speed, mem, bw_intra, bw_inter;
    int gpn; /* GPUs per node */
} otype;

/* Per-sample cost of each layer on one GPU of a plan (seconds/sample).
 * Compute: the profiled fwd+bwd time of the whole global batch on a speed-1
 * GPU, divided by the batch, the type's speed and the tensor degree (compute
 * splits evenly over intra-stage GPUs, Sec. 3.3).  Tensor parallel: four ring
 * all-reduces per layer and microbatch of the layer's output, on the intra-
 * node link.  MoE all-to-all: tokens x hidden x 2 B on the inter-node link
 * whenever the layer is spread over more than one GPU.  Comm terms scale
 * with the grid's contention factor kappa.  Latency is volume / bandwidth
 * (Sec. 3.4). */
static void layer_costs(const ojob* jb, const otype* ty, double kappa, int dp, int tp, double* u)
{
    for (int l = 0; l < jb->L; ++l) {
        double v = (double)jb->t[l] / ((double)jb->Bg * ty->speed * (double)tp);
        if (tp > 1)
            v += kappa * 8.0 * (double)(tp - 1) / (double)tp * (double)jb->x[l] / ty->bw_intra;
        if (dp * tp > 1)
            v += kappa * (double)jb->a2a[l] / ty->bw_inter;
        u[l] = v;
    }
}

typedef struct {
    double T;        /* iteration time (s) */
    double mem_max;  /* largest per-GPU footprint over stages (bytes) */
    double s_max;    /* slowest stage, per sample (s) */
    int feasible;
} oplan;

/* Price plan (dp, tp, pp, m) with stage cuts c_1..c_{pp-1} over prefix U.
 *   b      = Bg / (dp m) samples per microbatch
 *   W_k    = b (U_{c_{k+1}} - U_{c_k})               stage time per microbatch
 *   p2p_k  = kappa 2 b x_{last layer of k} / B_pp    (k < pp-1) activation out +
 *                                                     gradient back
 *   AR_k   = kappa [dp>1] 2(dp-1)/dp (P_k/tp) / B_dp fp32 gradient ring all-reduce
 *   Mem_k  = 4 P_k/tp + min(m, pp-k) b A_k/tp        weights, grads, two Adam
 *                                                     moments + in-flight 1F1B
 *                                                     activations
 *   T      = sum_k (W_k + p2p_k) + (m-1) max_k W_k + max_k AR_k
 * Pipeline neighbours sit dp*tp ranks apart (tp innermost, then dp, then pp):
 * B_pp is the intra-node link only when the whole plan fits in one node; the
 * dp group uses the intra-node link when it fits inside one node. */
static oplan price_plan(const ojob* jb, const otype* ty, int n, double kappa,
                        int dp, int tp, int pp, int m, const double* U, const int* cuts)
{
    oplan r;
    int bound[ORACLE_MAX_L + 2];
    bound[0] = 0;
    for (int k = 1; k < pp; ++k) bound[k] = cuts[k - 1];
    bound[pp] = jb->L;

    double b = (double)jb->Bg / (double)(dp * m);
    double B_pp = (n <= ty->gpn) ? ty->bw_intra : ty->bw_inter;
    int grp = dp * tp;
    double B_dp = (grp <= ty->gpn && ty->gpn % grp == 0) ? ty->bw_intra : ty->bw_inter;

    double fill = 0.0, w_max = 0.0, ar_max = 0.0, mem_max = 0.0, s_max = 0.0;
    for (int k = 0; k < pp; ++k) {
        int lo = bound[k], hi = bound[k + 1];
        double S = seg(U, lo, hi);
        double W = b * S;
        double Pk = 0.0, Ak = 0.0;
        for (int l = lo; l < hi; ++l) { Pk += (double)jb->p[l]; Ak += (double)jb->a[l]; }
        double p2p = 0.0;
        if (k < pp - 1) p2p = kappa * 2.0 * b * (double)jb->x[hi - 1] / B_pp;
        double AR = 0.0;
        if (dp > 1) AR = kappa * 2.0 * (double)(dp - 1) / (double)dp * (Pk / (double)tp) / B_dp;
        int inflight = m < pp - k ? m : pp - k;
        double Mem = 4.0 * Pk / (double)tp + (double)inflight * b * Ak / (double)tp;
        fill += W + p2p;
        if (W > w_max) w_max = W;
        if (S > s_max) s_max = S;
        if (AR > ar_max) ar_max = AR;
        if (Mem > mem_max) mem_max = Mem;
    }
    r.T = fill + (double)(m - 1) * w_max + ar_max;
    r.mem_max = mem_max;
    r.s_max = s_max;
    r.feasible = (mem_max <= ty->mem) ? 1 : 0;
    return r;
}

static int build_views(int j, int g, const int32_t* off, const float* t, const float* p,
                       const float* a, const float* x, const float* a2a, const int32_t* batch,
                       const float* speed, const float* mem, const float* bwi, const float* bwe,
                       const int32_t* gpn, ojob* jb, otype* ty)
{
    int s = off[j];
    jb->L = off[j + 1] - s;
    jb->Bg = batch[j];
    jb->t = t + s; jb->p = p + s; jb->a = a + s; jb->x = x + s; jb->a2a = a2a + s;
    ty->speed = speed[g]; ty->mem = mem[g]; ty->bw_intra = bwi[g]; ty->bw_inter = bwe[g];
    ty->gpn = gpn[g];
    return (jb->L >= 1 && jb->L <= ORACLE_MAX_L) ? 0 : -1;
}

/* ------------------------------------------------------------------ */
/* Exact-T stage partition                                             */
/* ------------------------------------------------------------------ */

/* The stages that minimise the plan's whole iteration time (Sec. 3.4: first
 * microbatch through every stage, B-1 more on the slowest, point-to-point
 * overlapped in the steady state; Eq. 4's once-per-iteration all-reduce).
 * The stage times summed over the stages are the same for every cut vector
 * (the stages tile the layers), so the cut-dependent part of T is
 *   Phi = (cS Smax + cX X) + cP Pmax, evaluated in that order, where
 *   Smax = max_k (U_{c_{k+1}} - U_{c_k})       slowest stage, per sample
 *   X    = x_{c_1 - 1} + (x_{c_2 - 1} + (... + x_{c_{pp-1} - 1}))   boundary bytes
 *   Pmax = max_k P_k                           largest stage's parameter bytes
 *   cS   = (m-1) b,   cX = kappa 2 b / B_pp,   cP = kappa 2 (dp-1) / dp / (tp B_dp)
 *          (cP = 0 when dp = 1), the coefficients of the steady state, the
 *          point-to-point fill and the all-reduce in the pricing.
 * Only cut vectors whose every stage fits memory count (the memory rule's
 * test, with a stage's parameter and activation bytes taken as differences of
 * the running totals over the layers).
 * Ties: the least (Phi, Smax, Pmax, X), then the lexicographically smallest
 * cut vector. */
typedef struct {
    const double* U;
    const omem* M;
    const double* x;        /* boundary activation bytes of each layer */
    int L, pp;
    double cS, cX, cP;
    double segP[ORACLE_MAX_L + 1][ORACLE_MAX_L + 1];   /* [lo][hi]: parameter bytes of [lo, hi) */
    double segA[ORACLE_MAX_L + 1][ORACLE_MAX_L + 1];   /* [lo][hi]: activation bytes per sample */
} oext;

typedef struct { double phi, s, p, x; } okey;

static int okey_less(const okey* a, const okey* b)
{
    if (a->phi != b->phi) return a->phi < b->phi;
    if (a->s != b->s) return a->s < b->s;
    if (a->p != b->p) return a->p < b->p;
    return a->x < b->x;
}

static double ext_phi(const oext* E, double sm, double x, double pm)
{
    return (E->cS * sm + E->cX * x) + E->cP * pm;
}

/* A stage's parameter and activation bytes under this rule: differences of
 * the running totals over the layers (summed left to right), like its cost. */
static void ext_tables(oext* E)
{
    double Pp[ORACLE_MAX_L + 1], Ap[ORACLE_MAX_L + 1];
    Pp[0] = 0.0;
    Ap[0] = 0.0;
    for (int l = 0; l < E->L; ++l) {
        Pp[l + 1] = Pp[l] + E->M->p[l];
        Ap[l + 1] = Ap[l] + E->M->a[l];
    }
    for (int lo = 0; lo <= E->L; ++lo)
        for (int hi = lo; hi <= E->L; ++hi) {
            E->segP[lo][hi] = Pp[hi] - Pp[lo];
            E->segA[lo][hi] = Ap[hi] - Ap[lo];
        }
}

/* Stage [lo, hi) as stage k (0-based) of pp fits memory (the memory rule's test). */
static int ext_fits(const oext* E, int lo, int hi, int k)
{
    return fits_sums(E->M, E->segP[lo][hi], E->segA[lo][hi], k, E->pp);
}

/* Brute force, the definition written out: every cut vector in lexicographic
 * order, the first with the least key among those whose stages all fit.
 * Returns Phi (+inf if none fits); cuts, key filled. */
typedef struct {
    const oext* E;
    int cur[ORACLE_MAX_L + 1];
    int best[ORACLE_MAX_L + 1];
    okey bkey;
    int found;
} oext_bf;

static void ext_bf_rec(oext_bf* b, int k)
{
    const oext* E = b->E;
    if (k == E->pp) {
        b->cur[k] = E->L;
        for (int q = 0; q < E->pp; ++q)
            if (!ext_fits(E, b->cur[q], b->cur[q + 1], q)) return;
        double sm = -INFINITY, pm = -INFINITY, x = 0.0;
        for (int q = 0; q < E->pp; ++q) {
            double sv = seg(E->U, b->cur[q], b->cur[q + 1]);
            double pv = E->segP[b->cur[q]][b->cur[q + 1]];
            if (sv > sm) sm = sv;
            if (pv > pm) pm = pv;
        }
        for (int q = E->pp - 1; q >= 1; --q) x = E->x[b->cur[q] - 1] + x;
        okey key = {ext_phi(E, sm, x, pm), sm, pm, x};
        if (!b->found || okey_less(&key, &b->bkey)) {
            b->bkey = key;
            b->found = 1;
            memcpy(b->best, b->cur, sizeof(int) * (size_t)(E->pp + 1));
        }
        return;
    }
    for (int c = b->cur[k - 1] + 1; c <= E->L - (E->pp - k); ++c) {
        b->cur[k] = c;
        ext_bf_rec(b, k + 1);
    }
}

static double exact_t_bruteforce(const oext* E, int* cuts, okey* key)
{
    oext_bf* b = (oext_bf*)xrealloc(NULL, sizeof(oext_bf));
    b->E = E;
    b->found = 0;
    b->cur[0] = 0;
    ext_bf_rec(b, 1);
    double phi = INFINITY;
    if (b->found) {
        phi = b->bkey.phi;
        if (key) *key = b->bkey;
        for (int k = 1; k < E->pp; ++k) cuts[k - 1] = b->best[k];
    }
    free(b);
    return phi;
}

/* Stage [i, e) allowed as stage k under the thresholds: its per-sample cost
 * at most tS, its parameter bytes at most tP, and it fits memory. */
static int ext_allowed(const oext* E, int i, int e, int k, double tS, double tP)
{
    return seg(E->U, i, e) <= tS && E->segP[i][e] <= tP && ext_fits(E, i, e, k);
}

/* Least X over the splits whose stages are all allowed, by a recursion over
 * suffixes: H[t][i] = least X of layers [i, L) as the last t stages (stage
 * pp - t first), with H[1][i] = 0 when [i, L) is allowed as the last stage and
 *   H[t][i] = min over e of x_{e-1} + H[t-1][e],  [i, e) allowed as stage pp-t.
 * (The sum is accumulated from the back, as X is defined.)  +inf if none. */
static double ext_xmin(const oext* E, double tS, double tP, double* H)
{
    int L = E->L, L1 = L + 1, pp = E->pp;
    for (int t = 0; t <= pp; ++t)
        for (int i = 0; i <= L; ++i) H[t * L1 + i] = INFINITY;
    for (int i = 0; i < L; ++i)
        if (ext_allowed(E, i, L, pp - 1, tS, tP)) H[1 * L1 + i] = 0.0;
    for (int t = 2; t <= pp; ++t)
        for (int i = 0; i <= L - t; ++i) {
            double best = INFINITY;
            for (int e = i + 1; e <= L - t + 1; ++e) {
                double h = H[(t - 1) * L1 + e];
                if (h == INFINITY || !ext_allowed(E, i, e, pp - t, tS, tP)) continue;
                double v = E->x[e - 1] + h;
                if (v < best) best = v;
            }
            H[t * L1 + i] = best;
        }
    return H[pp * L1 + 0];
}

/* Least largest stage value over the splits whose stages are allowed under
 * (tS, tP): F[t][i] = min over e of max(V(i, e), F[t-1][e]), F[1][i] = V(i, L),
 * as ext_xmin; V the stage's parameter bytes (which = 1) or its per-sample
 * cost (which = 0). */
static double ext_minmax(const oext* E, int which, double tS, double tP, double* F)
{
    int L = E->L, L1 = L + 1, pp = E->pp;
    for (int t = 0; t <= pp; ++t)
        for (int i = 0; i <= L; ++i) F[t * L1 + i] = INFINITY;
    for (int i = 0; i < L; ++i)
        if (ext_allowed(E, i, L, pp - 1, tS, tP)) F[1 * L1 + i] = which ? E->segP[i][L] : seg(E->U, i, L);
    for (int t = 2; t <= pp; ++t)
        for (int i = 0; i <= L - t; ++i) {
            double best = INFINITY;
            for (int e = i + 1; e <= L - t + 1; ++e) {
                double f = F[(t - 1) * L1 + e];
                if (f == INFINITY || !ext_allowed(E, i, e, pp - t, tS, tP)) continue;
                double vs = which ? E->segP[i][e] : seg(E->U, i, e);
                double v = vs > f ? vs : f;
                if (v < best) best = v;
            }
            F[t * L1 + i] = best;
        }
    return F[pp * L1 + 0];
}

static int cmp_double(const void* a, const void* b)
{
    double x = *(const double*)a, y = *(const double*)b;
    return (x > y) - (x < y);
}

/* Sorted distinct values of v[lo][hi] (0 <= lo < hi <= L) or of the U segments. */
static int ext_candidates(const oext* E, int which, double* out)
{
    int n = 0;
    for (int lo = 0; lo < E->L; ++lo)
        for (int hi = lo + 1; hi <= E->L; ++hi)
            out[n++] = which == 0 ? seg(E->U, lo, hi) : E->segP[lo][hi];
    qsort(out, (size_t)n, sizeof(double), cmp_double);
    int u = 0;
    for (int i = 0; i < n; ++i)
        if (u == 0 || out[i] != out[u - 1]) out[u++] = out[i];
    return u;
}

/* Exact-T by thresholds: for every pair (tS, tP) of a segment cost and a
 * segment parameter sum, the least X of the splits within them gives the key
 * ((cS tS + cX X) + cP tP, tS, tP, X); the least key over the pairs is the
 * least key over the splits (a split is counted at the pair of its own
 * maxima, and a pair's best split is no worse than the pair's key).  Pairs
 * are visited by tS, then tP, ascending; a pair after the best key found so
 * far in that order wins only with a smaller Phi, so the visit stops where a
 * lower bound of Phi reaches the best:
 *   tS runs from the least Smax of any split that fits; each tS stops the
 *   visit once (cS tS + cX Xlo) + cP Plo reaches the best (Xlo, Plo the least
 *   X and Pmax of any split that fits), or, when cS = 0, once the best equals
 *   the least Phi of any split;
 *   tP runs from the least Pmax of the splits within tS and stops once
 *   (cS tS + cX Xs) + cP tP reaches the best (Xs the least X within tS) or
 *   once its X is Xs.
 * The cuts are the lexicographically smallest split of least X within the
 * best pair, chosen left to right on the suffix table. */
static double exact_t(const oext* E, int* cuts, okey* key)
{
    int L = E->L, L1 = L + 1, pp = E->pp;
    size_t nc = (size_t)L * (size_t)(L + 1) / 2;
    double* cs = (double*)xrealloc(NULL, sizeof(double) * nc);
    double* cp = (double*)xrealloc(NULL, sizeof(double) * nc);
    double* H = (double*)xrealloc(NULL, sizeof(double) * (size_t)(pp + 1) * (size_t)L1);
    int ns = ext_candidates(E, 0, cs), np = ext_candidates(E, 1, cp);
    okey best = {INFINITY, INFINITY, INFINITY, INFINITY};
    int found = 0;
    double bs = 0.0, bp = 0.0;
    double p_lo = ext_minmax(E, 1, INFINITY, INFINITY, H);
    if (p_lo < INFINITY) {
        double s_lo = ext_minmax(E, 0, INFINITY, INFINITY, H);
        double x_lo = ext_xmin(E, INFINITY, INFINITY, H);
        /* cS = 0: the least Phi of any split, (cX X) + cP tP over tP */
        double phi_all = INFINITY;
        if (E->cS == 0.0) {
            for (int q = 0; q < np; ++q) {
                double tP = cp[q];
                if (tP < p_lo) continue;
                double X = ext_xmin(E, INFINITY, tP, H);
                if (X == INFINITY) continue;
                double v = (0.0 + E->cX * X) + E->cP * tP;
                if (v < phi_all) phi_all = v;
                if (X == x_lo) break;
            }
        }
        for (int a = 0; a < ns; ++a) {
            double tS = cs[a];
            if (tS < s_lo) continue;
            if (found && (E->cS == 0.0 ? best.phi <= phi_all : ext_phi(E, tS, x_lo, p_lo) >= best.phi)) break;
            double pmin = ext_minmax(E, 1, tS, INFINITY, H);
            if (pmin == INFINITY) continue;
            double xs = ext_xmin(E, tS, INFINITY, H);
            for (int q = 0; q < np; ++q) {
                double tP = cp[q];
                if (tP < pmin) continue;
                if (found && ext_phi(E, tS, xs, tP) >= best.phi) break;
                double X = ext_xmin(E, tS, tP, H);
                if (X == INFINITY) continue;
                okey k = {ext_phi(E, tS, X, tP), tS, tP, X};
                if (!found || okey_less(&k, &best)) {
                    best = k;
                    bs = tS;
                    bp = tP;
                    found = 1;
                }
                if (X == xs) break;
            }
        }
    }
    double phi = INFINITY;
    if (found) {
        phi = best.phi;
        if (key) *key = best;
        ext_xmin(E, bs, bp, H);
        int i = 0;
        for (int k = 1; k < pp; ++k) {
            int t = pp - k + 1, c = -1;
            for (int e = i + 1; e <= L - t + 1; ++e) {
                double h = H[(t - 1) * L1 + e];
                if (h == INFINITY || !ext_allowed(E, i, e, k - 1, bs, bp)) continue;
                if (E->x[e - 1] + h == H[t * L1 + i]) { c = e; break; }
            }
            if (c < 0) {
                fprintf(stderr, "arena oracle: exact-T cut reconstruction failed\n");
                abort();
            }
            cuts[k - 1] = c;
            i = c;
        }
    }
    free(cs);
    free(cp);
    free(H);
    return phi;
}

/* The coefficients of Phi for plan (dp, tp, pp, m) of a cell of n GPUs. */
static void ext_coefs(const ojob* jb, const otype* ty, int n, double kappa, int dp, int tp, int m, double* cS,
                      double* cX, double* cP)
{
    double b = (double)jb->Bg / (double)(dp * m);
    double B_pp = (n <= ty->gpn) ? ty->bw_intra : ty->bw_inter;
    int grp = dp * tp;
    double B_dp = (grp <= ty->gpn && ty->gpn % grp == 0) ? ty->bw_intra : ty->bw_inter;
    *cS = (double)(m - 1) * b;
    *cX = kappa * 2.0 * b / B_pp;
    *cP = dp > 1 ? kappa * 2.0 * (double)(dp - 1) / (double)dp / ((double)tp * B_dp) : 0.0;
}

/* Exposed for tests: the exact-T partition of one problem.  U: the per-sample
 * cost prefix; p, a, x: per-layer bytes; memory of the plan (m, b, tp, mem);
 * coefficients cS, cX, cP.  brute: enumerate every cut vector.  Returns Phi
 * (+inf if no split fits); cuts receives pp - 1 cuts and out[0..3] the key
 * (Phi, Smax, Pmax, X). */
double oracle_exact_t(const double* U, const double* p, const double* a, const double* x, int L, int pp,
                      int m, double b, int tp, double mem, double cS, double cX, double cP, int brute,
                      int* cuts, double* out)
{
    if (L < 1 || pp < 1 || pp > L || L > ORACLE_MAX_L || m < 1 || tp < 1) return NAN;
    omem M;
    M.p = p; M.a = a; M.L = L; M.m = m; M.tp = tp; M.b = b; M.mem = mem;
    oext* E = (oext*)xrealloc(NULL, sizeof(oext));
    E->U = U; E->M = &M; E->x = x; E->L = L; E->pp = pp; E->cS = cS; E->cX = cX; E->cP = cP;
    ext_tables(E);
    okey key = {INFINITY, INFINITY, INFINITY, INFINITY};
    double phi = brute ? exact_t_bruteforce(E, cuts, &key) : exact_t(E, cuts, &key);
    if (out) { out[0] = key.phi; out[1] = key.s; out[2] = key.p; out[3] = key.x; }
    free(E);
    return phi;
}

/* Price one plan of one cell.  If cuts_in is NULL the partition is the
 * canonical optimal one; otherwise cuts_in (pp-1 first-layer indices of
 * stages 1..pp-1) is priced as given.  out[0..3] = T, mem_max, s_max,
 * feasible; cuts_out (nullable) receives the cuts used.  Returns 0 on
 * success. */
/* The stage cuts of plan (dp, tp, pp, m) of a cell of n GPUs under partition
 * rule `rule`:
 * 0 = the canonical balanced partition (memory checked after pricing),
 * 1 = the canonical balanced partition among those whose every stage fits,
 * 2 = the exact-T partition (least iteration time among those that fit).
 * Returns 0, or -1 when rule 1 or 2 finds no split that fits. */
static int plan_cuts(const ojob* jb, const otype* ty, int rule, int n, double kappa, int dp, int tp, int pp,
                     int m, const double* U, int* cuts)
{
    if (rule == 0) {
        double W = oracle_bottleneck_dp(U, jb->L, pp);
        oracle_canonical_cuts(U, jb->L, pp, W, cuts);
        return 0;
    }
    double pd[ORACLE_MAX_L], ad[ORACLE_MAX_L], xd[ORACLE_MAX_L];
    for (int l = 0; l < jb->L; ++l) {
        pd[l] = (double)jb->p[l];
        ad[l] = (double)jb->a[l];
        xd[l] = (double)jb->x[l];
    }
    double b = (double)jb->Bg / (double)(dp * m);
    if (rule == 1) {
        omem M;
        M.p = pd; M.a = ad; M.L = jb->L; M.m = m; M.tp = tp;
        M.b = b;
        M.mem = ty->mem;
        return bottleneck_mem(U, &M, pp, cuts) < INFINITY ? 0 : -1;
    }
    double cS, cX, cP;
    ext_coefs(jb, ty, n, kappa, dp, tp, m, &cS, &cX, &cP);
    double phi = oracle_exact_t(U, pd, ad, xd, jb->L, pp, m, b, tp, ty->mem, cS, cX, cP, 0, cuts, NULL);
    return phi < INFINITY ? 0 : -1;
}

int oracle_eval_plan(int j, int g, int n, double kappa, int dp, int tp, int pp, int m,
                     const int32_t* off, const float* t, const float* p, const float* a,
                     const float* x, const float* a2a, const int32_t* batch,
                     const float* speed, const float* mem, const float* bwi, const float* bwe,
                     const int32_t* gpn, const int32_t* cuts_in, int32_t* cuts_out, double* out,
                     int rule)
{
    ojob jb; otype ty;
    if (build_views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, &jb, &ty)) return -1;
    if (dp < 1 || tp < 1 || pp < 1 || m < 1 || dp * tp * pp != n || pp > jb.L) return -1;
    if (rule < 0 || rule > 2) return -1;
    double u[ORACLE_MAX_L], U[ORACLE_MAX_L + 1];
    int cuts[ORACLE_MAX_L];
    layer_costs(&jb, &ty, kappa, dp, tp, u);
    oracle_prefix(u, jb.L, U);
    if (cuts_in) {
        for (int k = 0; k < pp - 1; ++k) {
            cuts[k] = cuts_in[k];
            int prevc = k == 0 ? 0 : cuts[k - 1];
            if (cuts[k] <= prevc || cuts[k] >= jb.L) return -1;
        }
    } else if (plan_cuts(&jb, &ty, rule, n, kappa, dp, tp, pp, m, U, cuts) != 0) {
        /* rule 1 or 2 and no split fits memory */
        out[0] = INFINITY; out[1] = INFINITY; out[2] = INFINITY; out[3] = 0.0;
        return 0;
    }
    oplan r = price_plan(&jb, &ty, n, kappa, dp, tp, pp, m, U, cuts);
    out[0] = r.T; out[1] = r.mem_max; out[2] = r.s_max; out[3] = (double)r.feasible;
    if (cuts_out)
        for (int k = 0; k < pp - 1; ++k) cuts_out[k] = cuts[k];
    return 0;
}

/* ------------------------------------------------------------------ */
/* Best plan of a cell                                                 */
/* ------------------------------------------------------------------ */

typedef struct {
    double T;
    int dp, tp, pp, m, feasible;
} ocand;

/* Lexicographic plan key: fewer stages, then less tensor parallelism, then
 * fewer microbatches. */
static int key_less(const ocand* a, const ocand* b)
{
    if (a->pp != b->pp) return a->pp < b->pp;
    if (a->tp != b->tp) return a->tp < b->tp;
    return a->m < b->m;
}

/* Enumerate every plan of cell (j, g, n): tp divides n and the node size,
 * pp divides n/tp and is at most the layer count, dp = n/(tp pp), and m is a
 * listed microbatch count with dp*m dividing the global batch (the global
 * batch is fixed under scaling, Sec. 3.5).  Each plan is priced with its
 * balanced partition under `rule` (see plan_cuts).  The cell's answer is the smallest (pp, tp, m) among
 * feasible plans whose T is within a factor (1 + tie_eps) of the smallest
 * feasible T.
 * res[0] = T (inf if none), res[1] = throughput (samples/s, 0 if none);
 * plan[0..3] = dp, tp, pp, m (0 if none); returns the number of plans
 * enumerated, or -1 on a bad job. */
int oracle_cell(int j, int g, int ci, const int32_t* off, const float* t, const float* p,
                const float* a, const float* x, const float* a2a, const int32_t* batch,
                const float* speed, const float* mem, const float* bwi, const float* bwe,
                const int32_t* gpn, const int32_t* counts, const float* kappa_grid, int n_counts,
                const int32_t* m_values, int n_m, double tie_eps,
                double* res, int32_t* plan, int32_t* cuts_out, int rule)
{
    ojob jb; otype ty;
    if (build_views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, &jb, &ty)) return -1;
    int n = counts[ci];
    double kappa = (double)kappa_grid[g * n_counts + ci];
    int L = jb.L;

    int cap = 64, nc = 0;
    ocand* cand = (ocand*)xrealloc(NULL, sizeof(ocand) * (size_t)cap);
    double u[ORACLE_MAX_L], U[ORACLE_MAX_L + 1];
    int cuts[ORACLE_MAX_L];

    for (int tp = 1; tp <= n; ++tp) {
        if (n % tp != 0 || tp > ty.gpn || ty.gpn % tp != 0) continue;
        for (int pp = 1; pp <= n / tp; ++pp) {
            if ((n / tp) % pp != 0 || pp > L) continue;
            int dp = n / (tp * pp);
            int any = 0;
            for (int mi = 0; mi < n_m; ++mi)
                if (jb.Bg % (dp * m_values[mi]) == 0) any = 1;
            if (!any) continue;
            layer_costs(&jb, &ty, kappa, dp, tp, u);
            oracle_prefix(u, L, U);
            /* the balanced partition does not depend on m: solved once per degree */
            if (rule == 0) plan_cuts(&jb, &ty, 0, n, kappa, dp, tp, pp, 1, U, cuts);
            for (int mi = 0; mi < n_m; ++mi) {
                int m = m_values[mi];
                if (jb.Bg % (dp * m) != 0) continue;
                if (nc == cap) { cap *= 2; cand = (ocand*)xrealloc(cand, sizeof(ocand) * (size_t)cap); }
                cand[nc].dp = dp; cand[nc].tp = tp; cand[nc].pp = pp; cand[nc].m = m;
                if (rule == 0 || plan_cuts(&jb, &ty, rule, n, kappa, dp, tp, pp, m, U, cuts) == 0) {
                    oplan r = price_plan(&jb, &ty, n, kappa, dp, tp, pp, m, U, cuts);
                    cand[nc].T = r.T;
                    cand[nc].feasible = r.feasible;
                } else {
                    cand[nc].T = INFINITY;
                    cand[nc].feasible = 0;
                }
                ++nc;
            }
        }
    }

    double tmin = INFINITY;
    for (int i = 0; i < nc; ++i)
        if (cand[i].feasible && cand[i].T < tmin) tmin = cand[i].T;
    int win = -1;
    if (tmin < INFINITY) {
        double lim = tmin * (1.0 + tie_eps);
        for (int i = 0; i < nc; ++i) {
            if (!cand[i].feasible || !(cand[i].T <= lim)) continue;
            if (win < 0 || key_less(&cand[i], &cand[win])) win = i;
        }
    }
    if (win < 0) {
        res[0] = INFINITY; res[1] = 0.0;
        plan[0] = plan[1] = plan[2] = plan[3] = 0;
    } else {
        ocand* w = &cand[win];
        res[0] = w->T;
        res[1] = (double)jb.Bg / w->T;
        plan[0] = w->dp; plan[1] = w->tp; plan[2] = w->pp; plan[3] = w->m;
        if (cuts_out) {
            layer_costs(&jb, &ty, kappa, w->dp, w->tp, u);
            oracle_prefix(u, L, U);
            plan_cuts(&jb, &ty, rule, n, kappa, w->dp, w->tp, w->pp, w->m, U, cuts);
            for (int k = 0; k < w->pp - 1; ++k) cuts_out[k] = cuts[k];
        }
    }
    free(cand);
    return nc;
}

/* Batch driver: evaluates the listed cells (flat index (j*T + g)*NC + ci).
 * res: 2 doubles per cell, plan: 4 ints per cell, cuts: cuts_stride ints
 * per cell (-1 past the last cut), nplans: plans enumerated per cell. */
int oracle_cells(int n_sel, const int64_t* cells, int n_types, int n_counts,
                 const int32_t* off, const float* t, const float* p, const float* a,
                 const float* x, const float* a2a, const int32_t* batch,
                 const float* speed, const float* mem, const float* bwi, const float* bwe,
                 const int32_t* gpn, const int32_t* counts, const float* kappa_grid,
                 const int32_t* m_values, int n_m, double tie_eps,
                 double* res, int32_t* plan, int32_t* cuts, int cuts_stride, int32_t* nplans,
                 int rule)
{
    if (rule < 0 || rule > 2) return -1;
    for (int s = 0; s < n_sel; ++s) {
        int64_t c = cells[s];
        int ci = (int)(c % n_counts);
        int g = (int)((c / n_counts) % n_types);
        int j = (int)(c / ((int64_t)n_counts * n_types));
        int32_t* crow = cuts ? cuts + (int64_t)s * cuts_stride : NULL;
        if (crow)
            for (int k = 0; k < cuts_stride; ++k) crow[k] = -1;
        int np = oracle_cell(j, g, ci, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn,
                             counts, kappa_grid, n_counts, m_values, n_m, tie_eps,
                             res + 2 * s, plan + 4 * s, crow, rule);
        if (np < 0) return -1;
        nplans[s] = np;
    }
    return 0;
}

/* Per-layer costs exposed for tests (same function the pricing uses). */
void oracle_layer_costs(int j, int g, double kappa, int dp, int tp,
                        const int32_t* off, const float* t, const float* p, const float* a,
                        const float* x, const float* a2a, const int32_t* batch,
                        const float* speed, const float* mem, const float* bwi, const float* bwe,
                        const int32_t* gpn, double* u)
{
    ojob jb; otype ty;
    if (build_views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, &jb, &ty)) return;
    layer_costs(&jb, &ty, kappa, dp, tp, u);
}

/* ------------------------------------------------------------------ */
/* Interpolated communication latency                                  */
/* ------------------------------------------------------------------ */

/* A communication primitive's latency is profiled at sampled volumes on the
 * target interconnect and interpolated by volume online (Sec. 3.4).  One
 * table per GPU type and link (0 inside a node, 1 across nodes): K points
 * vol[0] = 0 < vol[1] < ... < vol[K-1] bytes with latencies lat[k] seconds
 * (non-decreasing).  Nothing moved costs nothing; otherwise the latency is
 * linear between the samples around v and extended by the first or last
 * segment outside them. */
typedef struct {
    int K;
    const double* vol;
    const double* lat;
} otab;

static double tab_lat(const otab* tb, double v)
{
    if (!(v > 0.0)) return 0.0;
    int k = 1;
    while (k < tb->K - 1 && v > tb->vol[k]) ++k;
    return tb->lat[k - 1] + (v - tb->vol[k - 1]) * (tb->lat[k] - tb->lat[k - 1]) / (tb->vol[k] - tb->vol[k - 1]);
}

double oracle_tab_latency(int K, const double* vol, const double* lat, double v)
{
    otab tb;
    tb.K = K; tb.vol = vol; tb.lat = lat;
    return tab_lat(&tb, v);
}

/* Per-microbatch cost of each layer on one GPU of plan (dp, tp, m) with b
 * samples per microbatch: compute as in layer_costs times b; four tensor-
 * parallel ring all-reduces each moving 2 (tp-1)/tp b x_l bytes on the
 * intra-node link; the MoE all-to-all of b a2a_l bytes on the inter-node
 * link; communication scaled by kappa.  With a table linear through the
 * origin this is b times the per-sample cost of layer_costs. */
static void layer_costs_tab(const ojob* jb, const otype* ty, const otab* tabs, double kappa, int dp, int tp,
                            double b, double* c)
{
    for (int l = 0; l < jb->L; ++l) {
        double v = b * ((double)jb->t[l] / ((double)jb->Bg * ty->speed * (double)tp));
        if (tp > 1)
            v += kappa * (4.0 * tab_lat(&tabs[0], 2.0 * (double)(tp - 1) / (double)tp * b * (double)jb->x[l]));
        if (dp * tp > 1)
            v += kappa * tab_lat(&tabs[1], b * (double)jb->a2a[l]);
        c[l] = v;
    }
}

/* Price plan (dp, tp, pp, m) with stage cuts over the per-microbatch cost
 * prefix U:
 *   W_k   = U_{c_{k+1}} - U_{c_k}
 *   p2p_k = kappa 2 f_pp(b x_{last layer of k})      (k < pp-1), activation out
 *                                                     and gradient back
 *   AR_k  = kappa [dp>1] f_dp(2 (dp-1)/dp P_k/tp)     gradient ring all-reduce
 *   Mem_k as in price_plan
 *   T     = sum_k (W_k + p2p_k) + (m-1) max_k W_k + max_k AR_k
 * f_pp and f_dp are the tables of the links price_plan picks. */
static oplan price_plan_tab(const ojob* jb, const otype* ty, const otab* tabs, int n, double kappa,
                            int dp, int tp, int pp, int m, const double* U, const int* cuts)
{
    oplan r;
    int bound[ORACLE_MAX_L + 2];
    bound[0] = 0;
    for (int k = 1; k < pp; ++k) bound[k] = cuts[k - 1];
    bound[pp] = jb->L;

    double b = (double)jb->Bg / (double)(dp * m);
    const otab* t_pp = (n <= ty->gpn) ? &tabs[0] : &tabs[1];
    int grp = dp * tp;
    const otab* t_dp = (grp <= ty->gpn && ty->gpn % grp == 0) ? &tabs[0] : &tabs[1];

    double fill = 0.0, w_max = 0.0, ar_max = 0.0, mem_max = 0.0;
    for (int k = 0; k < pp; ++k) {
        int lo = bound[k], hi = bound[k + 1];
        double W = seg(U, lo, hi);
        double Pk = 0.0, Ak = 0.0;
        for (int l = lo; l < hi; ++l) { Pk += (double)jb->p[l]; Ak += (double)jb->a[l]; }
        double p2p = 0.0;
        if (k < pp - 1) p2p = kappa * (2.0 * tab_lat(t_pp, b * (double)jb->x[hi - 1]));
        double AR = 0.0;
        if (dp > 1) AR = kappa * tab_lat(t_dp, 2.0 * (double)(dp - 1) / (double)dp * (Pk / (double)tp));
        int inflight = m < pp - k ? m : pp - k;
        double Mem = 4.0 * Pk / (double)tp + (double)inflight * b * Ak / (double)tp;
        fill += W + p2p;
        if (W > w_max) w_max = W;
        if (AR > ar_max) ar_max = AR;
        if (Mem > mem_max) mem_max = Mem;
    }
    r.T = fill + (double)(m - 1) * w_max + ar_max;
    r.mem_max = mem_max;
    r.s_max = w_max;
    r.feasible = (mem_max <= ty->mem) ? 1 : 0;
    return r;
}

/* The tables of type g: tab[g][link] at vol/lat + (g*2 + link)*K. */
static void type_tabs(int g, int K, const double* vol, const double* lat, otab* tabs)
{
    for (int link = 0; link < 2; ++link) {
        tabs[link].K = K;
        tabs[link].vol = vol + ((size_t)g * 2 + (size_t)link) * (size_t)K;
        tabs[link].lat = lat + ((size_t)g * 2 + (size_t)link) * (size_t)K;
    }
}

/* Balanced partition of plan (dp, tp, pp, m) under the tables: its own
 * per-microbatch costs (they are no longer b times a per-sample cost, so
 * every microbatch count has its own partition), prefix, W* and canonical
 * cuts. */
static void plan_tab_partition(const ojob* jb, const otype* ty, const otab* tabs, double kappa, int dp, int tp,
                               int pp, int m, double* U, int* cuts)
{
    double c[ORACLE_MAX_L];
    double b = (double)jb->Bg / (double)(dp * m);
    layer_costs_tab(jb, ty, tabs, kappa, dp, tp, b, c);
    oracle_prefix(c, jb->L, U);
    double W = oracle_bottleneck_dp(U, jb->L, pp);
    oracle_canonical_cuts(U, jb->L, pp, W, cuts);
}

/* Price one plan under the tables (vol, lat: [T][2][K]); as oracle_eval_plan. */
int oracle_eval_plan_tab(int j, int g, int n, double kappa, int dp, int tp, int pp, int m,
                         const int32_t* off, const float* t, const float* p, const float* a,
                         const float* x, const float* a2a, const int32_t* batch,
                         const float* speed, const float* mem, const float* bwi, const float* bwe,
                         const int32_t* gpn, int K, const double* vol, const double* lat,
                         const int32_t* cuts_in, int32_t* cuts_out, double* out)
{
    ojob jb; otype ty;
    if (build_views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, &jb, &ty)) return -1;
    if (dp < 1 || tp < 1 || pp < 1 || m < 1 || dp * tp * pp != n || pp > jb.L || K < 2) return -1;
    otab tabs[2];
    type_tabs(g, K, vol, lat, tabs);
    double U[ORACLE_MAX_L + 1];
    int cuts[ORACLE_MAX_L];
    if (cuts_in) {
        double c[ORACLE_MAX_L];
        layer_costs_tab(&jb, &ty, tabs, kappa, dp, tp, (double)jb.Bg / (double)(dp * m), c);
        oracle_prefix(c, jb.L, U);
        for (int k = 0; k < pp - 1; ++k) {
            cuts[k] = cuts_in[k];
            int prevc = k == 0 ? 0 : cuts[k - 1];
            if (cuts[k] <= prevc || cuts[k] >= jb.L) return -1;
        }
    } else {
        plan_tab_partition(&jb, &ty, tabs, kappa, dp, tp, pp, m, U, cuts);
    }
    oplan r = price_plan_tab(&jb, &ty, tabs, n, kappa, dp, tp, pp, m, U, cuts);
    out[0] = r.T; out[1] = r.mem_max; out[2] = r.s_max; out[3] = (double)r.feasible;
    if (cuts_out)
        for (int k = 0; k < pp - 1; ++k) cuts_out[k] = cuts[k];
    return 0;
}

/* Best plan of cell (j, g, counts[ci]) under the tables: the plan space,
 * feasibility, tie window and key of oracle_cell; every plan priced with the
 * balanced partition of its own per-microbatch costs. */
static int oracle_cell_tab(int j, int g, int ci, const int32_t* off, const float* t, const float* p,
                           const float* a, const float* x, const float* a2a, const int32_t* batch,
                           const float* speed, const float* mem, const float* bwi, const float* bwe,
                           const int32_t* gpn, const int32_t* counts, const float* kappa_grid, int n_counts,
                           const int32_t* m_values, int n_m, double tie_eps, int K, const double* vol,
                           const double* lat, double* res, int32_t* plan, int32_t* cuts_out)
{
    ojob jb; otype ty;
    if (build_views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, &jb, &ty)) return -1;
    int n = counts[ci];
    double kappa = (double)kappa_grid[g * n_counts + ci];
    int L = jb.L;
    otab tabs[2];
    type_tabs(g, K, vol, lat, tabs);

    int cap = 64, nc = 0;
    ocand* cand = (ocand*)xrealloc(NULL, sizeof(ocand) * (size_t)cap);
    double U[ORACLE_MAX_L + 1];
    int cuts[ORACLE_MAX_L];
    for (int tp = 1; tp <= n; ++tp) {
        if (n % tp != 0 || tp > ty.gpn || ty.gpn % tp != 0) continue;
        for (int pp = 1; pp <= n / tp; ++pp) {
            if ((n / tp) % pp != 0 || pp > L) continue;
            int dp = n / (tp * pp);
            for (int mi = 0; mi < n_m; ++mi) {
                int m = m_values[mi];
                if (jb.Bg % (dp * m) != 0) continue;
                plan_tab_partition(&jb, &ty, tabs, kappa, dp, tp, pp, m, U, cuts);
                oplan r = price_plan_tab(&jb, &ty, tabs, n, kappa, dp, tp, pp, m, U, cuts);
                if (nc == cap) { cap *= 2; cand = (ocand*)xrealloc(cand, sizeof(ocand) * (size_t)cap); }
                cand[nc].T = r.T; cand[nc].dp = dp; cand[nc].tp = tp; cand[nc].pp = pp;
                cand[nc].m = m; cand[nc].feasible = r.feasible;
                ++nc;
            }
        }
    }
    double tmin = INFINITY;
    for (int i = 0; i < nc; ++i)
        if (cand[i].feasible && cand[i].T < tmin) tmin = cand[i].T;
    int win = -1;
    if (tmin < INFINITY) {
        double lim = tmin * (1.0 + tie_eps);
        for (int i = 0; i < nc; ++i) {
            if (!cand[i].feasible || !(cand[i].T <= lim)) continue;
            if (win < 0 || key_less(&cand[i], &cand[win])) win = i;
        }
    }
    if (win < 0) {
        res[0] = INFINITY; res[1] = 0.0;
        plan[0] = plan[1] = plan[2] = plan[3] = 0;
    } else {
        ocand* w = &cand[win];
        res[0] = w->T;
        res[1] = (double)jb.Bg / w->T;
        plan[0] = w->dp; plan[1] = w->tp; plan[2] = w->pp; plan[3] = w->m;
        if (cuts_out) {
            plan_tab_partition(&jb, &ty, tabs, kappa, w->dp, w->tp, w->pp, w->m, U, cuts);
            for (int k = 0; k < w->pp - 1; ++k) cuts_out[k] = cuts[k];
        }
    }
    free(cand);
    return nc;
}

/* Batch driver under the tables (vol, lat: [n_types][2][K]); as oracle_cells. */
int oracle_cells_tab(int n_sel, const int64_t* cells, int n_types, int n_counts,
                     const int32_t* off, const float* t, const float* p, const float* a,
                     const float* x, const float* a2a, const int32_t* batch,
                     const float* speed, const float* mem, const float* bwi, const float* bwe,
                     const int32_t* gpn, const int32_t* counts, const float* kappa_grid,
                     const int32_t* m_values, int n_m, double tie_eps, int K, const double* vol,
                     const double* lat, double* res, int32_t* plan, int32_t* cuts, int cuts_stride,
                     int32_t* nplans)
{
    if (K < 2) return -1;
    for (int s = 0; s < n_sel; ++s) {
        int64_t c = cells[s];
        int ci = (int)(c % n_counts);
        int g = (int)((c / n_counts) % n_types);
        int j = (int)(c / ((int64_t)n_counts * n_types));
        int32_t* crow = cuts ? cuts + (int64_t)s * cuts_stride : NULL;
        if (crow)
            for (int k = 0; k < cuts_stride; ++k) crow[k] = -1;
        int np = oracle_cell_tab(j, g, ci, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn,
                                 counts, kappa_grid, n_counts, m_values, n_m, tie_eps, K, vol, lat,
                                 res + 2 * s, plan + 4 * s, crow);
        if (np < 0) return -1;
        nplans[s] = np;
    }
    return 0;
}
