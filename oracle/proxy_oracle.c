/*
 * CPU oracle of the proxy-plan planner: TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite and the benchmark's CPU-baseline leg may load this
 * library.  The product path never calls it; it shares no code, header,
 * table or constant with the HIP library.
 *
 * For one (job, GPU type, GPU count) cell it follows the load-aware planner
 * of Sec. 3.3 step by step, plainly and slowly, in IEEE double precision
 * from the f32 input tables:
 *
 *   1. the job's layers form O = min(L, n_ops) clustered operators
 *      (operator i holds layers floor(iL/O) .. floor((i+1)L/O) - 1);
 *   2. each operator's load by the roofline (Eq. 2): FLOPs = f_ref * sum t,
 *      memory traffic = sum (p + Bg a); load = max(FLOPs / (speed f_ref),
 *      traffic / HBM bandwidth), the time form of FLOPs / R(FLOPs / Mem);
 *   3. its proportional GPU share d_i = (load_i / sum load) n;
 *   4. for every pipeline degree s (a grid of Sec. 3.2) every contiguous
 *      grouping of the O operators into s stages, stage share D_j = sum d_i;
 *   5. the power-of-two normalisation minimising the computation bias
 *      (Eq. 3): stage counts that are powers of two summing to n;
 *   6. for each microbatch count B, per stage the intra-stage plan (dp, tp)
 *      with the least communication within the memory limit, and the
 *      communication load l_comm (Eq. 4);
 *   7. the proxy plan of the grid (s, B): least computation bias, then least
 *      communication load (the lexicographic minimum, always a member of the
 *      Pareto frontier of the two metrics);
 *   8. each grid's proxy priced by the 1F1B model (Sec. 3.4), generalised to
 *      per-stage GPU counts, and the best grid of the cell.
 *
 * The readings where the paper leaves a step open (P1-P12) are listed in the
 * repository's design notes; each function names the ones it follows.
 *
 * Pins (tests/test_oracle_proxy.py): the normalisation against brute force
 * over every ordered power-of-two vector, the enumeration against an
 * independent one, the pricing against the uniform-plan oracle when every
 * stage is alike, hand-derived loads, l_comm and intra-stage choices.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PO_MAX_OPS 16
#define PO_MAX_L 128
#define PO_MAX_M 16                 /* microbatch counts per call */

typedef struct {
    int L, Bg;
    const float *t, *p, *a, *x, *a2a;
} pjob;

typedef struct {
    double speed, mem, bw_intra, bw_inter, hbm;
    int gpn;
} ptype;

/* Operator sums (P1): every sum runs over the operator's layers left to
 * right. */
typedef struct {
    int O;
    int lo[PO_MAX_OPS + 1];          /* first layer of operator i; lo[O] = L */
    double T[PO_MAX_OPS];            /* sum t */
    double X[PO_MAX_OPS];            /* sum x (tensor-parallel all-reduce volume per sample) */
    double E[PO_MAX_OPS];            /* sum a2a (all-to-all volume per sample) */
    double P[PO_MAX_OPS];            /* sum p (parameter bytes) */
    double A[PO_MAX_OPS];            /* sum a (stored activation bytes per sample) */
    double M[PO_MAX_OPS];            /* sum (p + Bg a): memory traffic for the global batch */
    double xlast[PO_MAX_OPS];        /* x of the operator's last layer (pipeline boundary) */
    double load[PO_MAX_OPS];         /* Eq. 2 */
    double d[PO_MAX_OPS];            /* proportional GPU share */
    double lsum;                     /* total load; a job without any has no proxy plan */
} pops;

static void build_ops(const pjob* jb, const ptype* ty, double f_ref, int n_ops, int n, pops* o)
{
    int O = jb->L < n_ops ? jb->L : n_ops;
    o->O = O;
    for (int i = 0; i <= O; ++i) o->lo[i] = (int)(((long long)i * jb->L) / O);
    double lsum = 0.0;
    for (int i = 0; i < O; ++i) {
        double T = 0.0, X = 0.0, E = 0.0, P = 0.0, A = 0.0, M = 0.0;
        for (int l = o->lo[i]; l < o->lo[i + 1]; ++l) {
            T += (double)jb->t[l];
            X += (double)jb->x[l];
            E += (double)jb->a2a[l];
            P += (double)jb->p[l];
            A += (double)jb->a[l];
            M += (double)jb->p[l] + (double)jb->Bg * (double)jb->a[l];
        }
        o->T[i] = T; o->X[i] = X; o->E[i] = E; o->P[i] = P; o->A[i] = A; o->M[i] = M;
        o->xlast[i] = (double)jb->x[o->lo[i + 1] - 1];
        /* Eq. 2: FLOPs / R(FLOPs / Mem), R the roofline of the type */
        double flops = f_ref * T;
        double compute = flops / (ty->speed * f_ref);
        double memory = M / ty->hbm;
        o->load[i] = compute > memory ? compute : memory;
        lsum += o->load[i];
    }
    o->lsum = lsum;
    for (int i = 0; i < O; ++i) o->d[i] = (o->load[i] / lsum) * (double)n;
}

/* ------------------------------------------------------------------ */
/* Power-of-two normalisation (Eq. 3, readings P5-P6)                  */
/* ------------------------------------------------------------------ */

typedef struct {
    int s, n;
    double D[PO_MAX_OPS];     /* stage shares in stage order */
    int ord[PO_MAX_OPS];      /* stages by share, largest first (ties: lower stage first) */
    int pos[PO_MAX_OPS];      /* sorted position of each stage (inverse of ord) */
    int cur[PO_MAX_OPS];      /* exponents being tried, sorted position order */
    int best[PO_MAX_OPS];
    double best_cost;
    int found;
} pnorm;

/* lexicographic comparison of two exponent sequences, larger first wins */
static int lex_greater(const int* a, const int* b, int s)
{
    for (int k = 0; k < s; ++k) {
        if (a[k] != b[k]) return a[k] > b[k];
    }
    return 0;
}

/* Every multiset of powers of two (non-increasing exponents, at most maxe),
 * paired with the shares in sorted order (the largest count to the largest
 * share); the squared bias is accumulated over the stages in stage order. */
static void norm_rec(pnorm* st, int k, int remaining, int maxe)
{
    if (k == st->s) {
        if (remaining != 0) return;
        double cost = 0.0;
        for (int j = 0; j < st->s; ++j) {
            double diff = (double)(1 << st->cur[st->pos[j]]) - st->D[j];
            cost += diff * diff;
        }
        if (!st->found || cost < st->best_cost ||
            (cost == st->best_cost && lex_greater(st->cur, st->best, st->s))) {
            st->found = 1;
            st->best_cost = cost;
            memcpy(st->best, st->cur, sizeof(int) * st->s);
        }
        return;
    }
    int left = st->s - k - 1;        /* stages after this one need at least 1 GPU each */
    for (int e = maxe; e >= 0; --e) {
        int v = 1 << e;
        if (v > remaining - left) continue;
        if ((long long)(left + 1) * v < remaining) break;   /* later stages take at most v each */
        st->cur[k] = e;
        norm_rec(st, k + 1, remaining - v, e);
    }
}

/* The normalised counts m_out (stage order) minimising the bias, and the
 * squared bias; returns -1 if no s powers of two sum to n.  For a given
 * multiset the sorted pairing is the best assignment (rearrangement
 * inequality), so the search runs over multisets.  Ties: the
 * lexicographically larger sorted multiset. */
double proxy_oracle_normalize(const double* D, int s, int n, int32_t* m_out)
{
    pnorm st;
    memset(&st, 0, sizeof(st));
    st.s = s;
    st.n = n;
    for (int j = 0; j < s; ++j) st.D[j] = D[j];
    for (int j = 0; j < s; ++j) {              /* stable insertion sort, largest share first */
        int q = j;
        while (q > 0 && st.D[st.ord[q - 1]] < D[j]) {
            st.ord[q] = st.ord[q - 1];
            --q;
        }
        st.ord[q] = j;
    }
    for (int q = 0; q < s; ++q) st.pos[st.ord[q]] = q;

    int maxe = 0;
    while ((1 << (maxe + 1)) <= n) ++maxe;
    norm_rec(&st, 0, n, maxe);
    if (!st.found) return -1.0;
    for (int q = 0; q < s; ++q) m_out[st.ord[q]] = 1 << st.best[q];
    return st.best_cost;
}

/* ------------------------------------------------------------------ */
/* Stage terms of a plan with per-stage GPU counts (readings P7-P10)    */
/* ------------------------------------------------------------------ */

typedef struct {
    int s, B;
    int bound[PO_MAX_OPS + 1];       /* stage j holds operators bound[j] .. bound[j+1]-1 */
    int Dn[PO_MAX_OPS];              /* GPUs of stage j (powers of two) */
    int tp[PO_MAX_OPS];              /* intra-stage tensor degree */
} pplan;

typedef struct {
    double T, lcomm;
    int feasible;
} pprice;

static double stage_sum(const double* v, int lo, int hi)
{
    double s = 0.0;
    for (int i = lo; i < hi; ++i) s += v[i];
    return s;
}

/* Per-microbatch samples of one replica of stage j, or a negative value if
 * dp B does not divide the batch. */
static double replica_batch(const pjob* jb, int D, int tp, int B)
{
    int dp = D / tp;
    if (jb->Bg % (dp * B)) return -1.0;
    return (double)jb->Bg / (double)(dp * B);
}

/* Intra-stage communication of stage j per microbatch (tensor-parallel
 * all-reduces and MoE all-to-all, reading P7) and its gradient all-reduce
 * per iteration, for (D, tp). */
static void stage_comm(const pjob* jb, const ptype* ty, const pops* o, double kappa, int lo, int hi,
                       int D, int tp, double b, double* C, double* AR)
{
    double X = stage_sum(o->X, lo, hi), E = stage_sum(o->E, lo, hi), P = stage_sum(o->P, lo, hi);
    double per_sample = 0.0;
    if (tp > 1) per_sample += kappa * 8.0 * (double)(tp - 1) / (double)tp * X / ty->bw_intra;
    if (D > 1) per_sample += kappa * E / ty->bw_inter;
    *C = b * per_sample;
    int dp = D / tp;
    double B_dp = (D <= ty->gpn && ty->gpn % D == 0) ? ty->bw_intra : ty->bw_inter;
    *AR = 0.0;
    if (dp > 1) *AR = kappa * 2.0 * (double)(dp - 1) / (double)dp * (P / (double)tp) / B_dp;
    (void)jb;
}

static double stage_mem(const pops* o, int lo, int hi, int tp, double b, int inflight)
{
    double P = stage_sum(o->P, lo, hi), A = stage_sum(o->A, lo, hi);
    return 4.0 * P / (double)tp + (double)inflight * b * A / (double)tp;
}

/* The stage's intra-stage plan: tp a power of two dividing both its GPU count
 * and the node size, dp = D / tp with dp B dividing the batch, within the
 * memory limit; least communication per iteration B C + AR; ties: smaller tp.
 * Returns the tp, or 0 if none fits. */
static int choose_tp(const pjob* jb, const ptype* ty, const pops* o, double kappa, int lo, int hi,
                     int D, int B, int inflight)
{
    int best = 0;
    double best_cost = 0.0;
    for (int tp = 1; tp <= D; tp *= 2) {
        if (D % tp || ty->gpn % tp) continue;
        double b = replica_batch(jb, D, tp, B);
        if (b < 0.0) continue;
        if (stage_mem(o, lo, hi, tp, b, inflight) > ty->mem) continue;
        double C, AR;
        stage_comm(jb, ty, o, kappa, lo, hi, D, tp, b, &C, &AR);
        double cost = (double)B * C + AR;
        if (best == 0 || cost < best_cost) {
            best = tp;
            best_cost = cost;
        }
    }
    return best;
}

/* Chooses every stage's tp (P7) and evaluates l_comm (Eq. 4, reading P8):
 * (B - 1) max_j C_j + sum_j C_j + sum_j AR_j.  Returns 0 if some stage has
 * no intra-stage plan that fits. */
static int plan_lcomm(const pjob* jb, const ptype* ty, const pops* o, double kappa, pplan* pl, double* lcomm)
{
    double cmax = 0.0, csum = 0.0, arsum = 0.0;
    for (int j = 0; j < pl->s; ++j) {
        int lo = pl->bound[j], hi = pl->bound[j + 1];
        int inflight = pl->B < pl->s - j ? pl->B : pl->s - j;
        int tp = choose_tp(jb, ty, o, kappa, lo, hi, pl->Dn[j], pl->B, inflight);
        if (tp == 0) return 0;
        pl->tp[j] = tp;
        double b = replica_batch(jb, pl->Dn[j], tp, pl->B);
        double C, AR;
        stage_comm(jb, ty, o, kappa, lo, hi, pl->Dn[j], tp, b, &C, &AR);
        if (C > cmax) cmax = C;
        csum += C;
        arsum += AR;
    }
    *lcomm = (double)(pl->B - 1) * cmax + csum + arsum;
    return 1;
}

/* The 1F1B iteration time of a plan with per-stage (dp_j, tp_j) (reading
 * P10): W_j = b_j (T_j / (Bg speed tp_j) + comm per sample), b_j = Bg /
 * (dp_j B); p2p between stages j and j+1 carries 2 x_last Bg / (B min(dp_j,
 * dp_j+1)) bytes; AR_j the gradient all-reduce; memory per stage as in the
 * uniform model; T = sum_j (W_j + p2p_j) + (B-1) max_j W_j + max_j AR_j. */
static pprice price(const pjob* jb, const ptype* ty, const pops* o, double kappa, int n, const pplan* pl)
{
    pprice r;
    r.feasible = 1;
    r.lcomm = 0.0;
    double B_pp = (n <= ty->gpn) ? ty->bw_intra : ty->bw_inter;
    double fill = 0.0, wmax = 0.0, armax = 0.0;
    for (int j = 0; j < pl->s; ++j) {
        int lo = pl->bound[j], hi = pl->bound[j + 1];
        int D = pl->Dn[j], tp = pl->tp[j], dp = D / tp;
        double b = replica_batch(jb, D, tp, pl->B);
        if (b < 0.0) { r.feasible = 0; r.T = INFINITY; return r; }
        int inflight = pl->B < pl->s - j ? pl->B : pl->s - j;
        if (stage_mem(o, lo, hi, tp, b, inflight) > ty->mem) r.feasible = 0;
        double T = stage_sum(o->T, lo, hi), X = stage_sum(o->X, lo, hi), E = stage_sum(o->E, lo, hi);
        double P = stage_sum(o->P, lo, hi);
        double per_sample = T / ((double)jb->Bg * ty->speed * (double)tp);
        if (tp > 1) per_sample += kappa * 8.0 * (double)(tp - 1) / (double)tp * X / ty->bw_intra;
        if (D > 1) per_sample += kappa * E / ty->bw_inter;
        double W = b * per_sample;
        double p2p = 0.0;
        if (j < pl->s - 1) {
            int dpn = pl->Dn[j + 1] / pl->tp[j + 1];
            int dmin = dp < dpn ? dp : dpn;
            p2p = kappa * 2.0 * ((double)jb->Bg / (double)(dmin * pl->B)) * o->xlast[hi - 1] / B_pp;
        }
        double B_dp = (D <= ty->gpn && ty->gpn % D == 0) ? ty->bw_intra : ty->bw_inter;
        double AR = 0.0;
        if (dp > 1) AR = kappa * 2.0 * (double)(dp - 1) / (double)dp * (P / (double)tp) / B_dp;
        fill += W + p2p;
        if (W > wmax) wmax = W;
        if (AR > armax) armax = AR;
    }
    r.T = fill + (double)(pl->B - 1) * wmax + armax;
    if (!r.feasible) r.T = INFINITY;
    return r;
}

/* ------------------------------------------------------------------ */
/* Proxy plan of one grid and the best grid of a cell                   */
/* ------------------------------------------------------------------ */

typedef struct {
    int ok;
    double b2, lcomm, T;
    pplan pl;
} pgrid;

typedef struct {
    const pjob* jb;
    const ptype* ty;
    const pops* o;
    double kappa;
    int n, s, n_m;
    const int32_t* m_values;
    int cut[PO_MAX_OPS];             /* operator index where stage k+1 starts */
    pgrid best[PO_MAX_M];            /* the proxy of grid (s, m_values[k]) so far */
} penum;

/* Every grouping of the operators into s stages, cut vectors in
 * lexicographic order; the first one seen wins exact ties.  The
 * normalisation does not depend on B, so it is done once per grouping and
 * each B then takes its own intra-stage plans and l_comm. */
static void enum_rec(penum* e, int k, int start)
{
    int s = e->s, O = e->o->O;
    if (k == s - 1) {
        pplan pl;
        pl.s = s;
        pl.bound[0] = 0;
        for (int q = 0; q < s - 1; ++q) pl.bound[q + 1] = e->cut[q];
        pl.bound[s] = O;
        double D[PO_MAX_OPS] = {0.0};
        for (int j = 0; j < s; ++j) D[j] = stage_sum(e->o->d, pl.bound[j], pl.bound[j + 1]);
        int32_t m[PO_MAX_OPS];
        double b2 = proxy_oracle_normalize(D, s, e->n, m);
        if (b2 < 0.0) return;
        for (int j = 0; j < s; ++j) pl.Dn[j] = m[j];
        for (int q = 0; q < e->n_m; ++q) {
            pgrid* bq = &e->best[q];
            if (bq->ok && b2 > bq->b2) continue;       /* cannot be the proxy of this grid */
            pl.B = e->m_values[q];
            double lcomm;
            if (!plan_lcomm(e->jb, e->ty, e->o, e->kappa, &pl, &lcomm)) continue;   /* does not fit */
            if (!bq->ok || b2 < bq->b2 || (b2 == bq->b2 && lcomm < bq->lcomm)) {
                bq->ok = 1;
                bq->b2 = b2;
                bq->lcomm = lcomm;
                bq->pl = pl;
            }
        }
        return;
    }
    /* stage k+1 starts at operator c; leave at least one operator per later stage */
    for (int c = start + 1; c <= O - (s - 1 - k); ++c) {
        e->cut[k] = c;
        enum_rec(e, k + 1, c);
    }
}

/* The proxies of the grids (s, B) for every B in m_values, priced. */
static void grid_proxies(const pjob* jb, const ptype* ty, const pops* o, double kappa, int n, int s,
                         const int32_t* m_values, int n_m, pgrid* out)
{
    penum e;
    memset(&e, 0, sizeof(e));
    e.jb = jb; e.ty = ty; e.o = o; e.kappa = kappa; e.n = n; e.s = s;
    e.m_values = m_values; e.n_m = n_m;
    if (o->lsum > 0.0) enum_rec(&e, 0, 0);      /* zero total load: no shares, no proxy */
    for (int q = 0; q < n_m; ++q) {
        out[q] = e.best[q];
        if (out[q].ok) {
            pprice pr = price(jb, ty, o, kappa, n, &out[q].pl);
            out[q].T = pr.T;
            if (!pr.feasible) out[q].ok = 0;
        }
    }
}

static int views(int j, int g, const int32_t* off, const float* t, const float* p, const float* a,
                 const float* x, const float* a2a, const int32_t* batch, const float* speed,
                 const float* mem, const float* bwi, const float* bwe, const int32_t* gpn,
                 const float* hbm, pjob* jb, ptype* ty)
{
    int s0 = off[j];
    jb->L = off[j + 1] - s0;
    jb->Bg = batch[j];
    jb->t = t + s0; jb->p = p + s0; jb->a = a + s0; jb->x = x + s0; jb->a2a = a2a + s0;
    ty->speed = speed[g]; ty->mem = mem[g]; ty->bw_intra = bwi[g]; ty->bw_inter = bwe[g];
    ty->gpn = gpn[g]; ty->hbm = hbm[g];
    return (jb->L >= 1 && jb->L <= PO_MAX_L) ? 0 : -1;
}

/* Per-operator loads and GPU shares of a job on a type with n GPUs:
 * out[0..O-1] = load, out[O..2O-1] = d.  Returns O. */
int proxy_oracle_loads(int j, int g, int n, const int32_t* off, const float* t, const float* p,
                       const float* a, const float* x, const float* a2a, const int32_t* batch,
                       const float* speed, const float* mem, const float* bwi, const float* bwe,
                       const int32_t* gpn, const float* hbm, double f_ref, int n_ops, double* out)
{
    pjob jb; ptype ty; pops o;
    if (views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, hbm, &jb, &ty)) return -1;
    build_ops(&jb, &ty, f_ref, n_ops, n, &o);
    for (int i = 0; i < o.O; ++i) { out[i] = o.load[i]; out[o.O + i] = o.d[i]; }
    return o.O;
}

/* Price a given plan: stage boundaries at operators (bounds[0..s], bounds[0]
 * = 0, bounds[s] = O), GPUs and tp per stage, B microbatches.  out = T,
 * feasible, l_comm (with the given tps). */
int proxy_oracle_price(int j, int g, int n, double kappa, int s, int B, const int32_t* bounds,
                       const int32_t* Dn, const int32_t* tp, const int32_t* off, const float* t,
                       const float* p, const float* a, const float* x, const float* a2a,
                       const int32_t* batch, const float* speed, const float* mem, const float* bwi,
                       const float* bwe, const int32_t* gpn, const float* hbm, double f_ref, int n_ops,
                       double* out)
{
    pjob jb; ptype ty; pops o;
    if (views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, hbm, &jb, &ty)) return -1;
    build_ops(&jb, &ty, f_ref, n_ops, n, &o);
    if (s < 1 || s > o.O) return -1;
    pplan pl;
    pl.s = s;
    pl.B = B;
    for (int q = 0; q <= s; ++q) pl.bound[q] = bounds[q];
    if (pl.bound[0] != 0 || pl.bound[s] != o.O) return -1;
    for (int q = 0; q < s; ++q) {
        if (pl.bound[q + 1] <= pl.bound[q]) return -1;
        pl.Dn[q] = Dn[q];
        pl.tp[q] = tp[q];
        if (Dn[q] < 1 || tp[q] < 1 || Dn[q] % tp[q]) return -1;
    }
    pprice pr = price(&jb, &ty, &o, kappa, n, &pl);
    double cmax = 0.0, csum = 0.0, arsum = 0.0;
    for (int q = 0; q < s; ++q) {
        double b = replica_batch(&jb, pl.Dn[q], pl.tp[q], B);
        if (b < 0.0) { csum = INFINITY; break; }
        double C, AR;
        stage_comm(&jb, &ty, &o, kappa, pl.bound[q], pl.bound[q + 1], pl.Dn[q], pl.tp[q], b, &C, &AR);
        if (C > cmax) cmax = C;
        csum += C;
        arsum += AR;
    }
    out[0] = pr.T;
    out[1] = (double)pr.feasible;
    out[2] = (double)(B - 1) * cmax + csum + arsum;
    return 0;
}

/* The proxy plan of one grid (s, B) of a cell.  out = ok, b2, l_comm, T;
 * plan[0..s] = stage bounds (operators), plan[17..17+s-1] = GPUs per stage,
 * plan[33..33+s-1] = tp per stage. */
int proxy_oracle_grid(int j, int g, int n, double kappa, int s, int B, const int32_t* off,
                      const float* t, const float* p, const float* a, const float* x,
                      const float* a2a, const int32_t* batch, const float* speed, const float* mem,
                      const float* bwi, const float* bwe, const int32_t* gpn, const float* hbm,
                      double f_ref, int n_ops, double* out, int32_t* plan)
{
    pjob jb; ptype ty; pops o;
    if (views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, hbm, &jb, &ty)) return -1;
    build_ops(&jb, &ty, f_ref, n_ops, n, &o);
    if (s < 1 || s > o.O || s > n || B < 1) return -1;
    int32_t mv[1] = {B};
    pgrid r;
    grid_proxies(&jb, &ty, &o, kappa, n, s, mv, 1, &r);
    out[0] = r.ok; out[1] = r.b2; out[2] = r.lcomm; out[3] = r.ok ? r.T : INFINITY;
    for (int q = 0; q < 49; ++q) plan[q] = 0;
    if (r.ok) {
        for (int q = 0; q <= s; ++q) plan[q] = r.pl.bound[q];
        for (int q = 0; q < s; ++q) { plan[17 + q] = r.pl.Dn[q]; plan[33 + q] = r.pl.tp[q]; }
    }
    return 0;
}

/* The proxy-estimated best plan of cells (j, g, ci), cell id (j T + g) NC +
 * ci: every grid (s = 1..min(O, n), B in m_values) gets its proxy, priced by
 * the 1F1B model; the least T wins, T within (1 + tie_eps) of the least
 * counting as a tie, broken by fewer stages, then fewer microbatches
 * (reading P11).  out[4 c ..] = T (inf if no grid fits), b2, l_comm, Bg/T;
 * plan[52 c ..] = s, B, bounds[0..s] at 2.., GPUs per stage at 19.., tp per
 * stage at 35.. (zero when infeasible). */
int proxy_oracle_cells(int n_sel, const int64_t* cells, int n_types, int n_counts, const int32_t* off,
                       const float* t, const float* p, const float* a, const float* x, const float* a2a,
                       const int32_t* batch, const float* speed, const float* mem, const float* bwi,
                       const float* bwe, const int32_t* gpn, const float* hbm, const int32_t* counts,
                       const float* kappa, const int32_t* m_values, int n_m, double tie_eps, double f_ref,
                       int n_ops, double* out, int32_t* plan)
{
    for (int q = 0; q < n_sel; ++q) {
        int64_t c = cells[q];
        int ci = (int)(c % n_counts);
        int g = (int)((c / n_counts) % n_types);
        int j = (int)(c / ((int64_t)n_counts * n_types));
        int n = counts[ci];
        double kap = (double)kappa[(int64_t)g * n_counts + ci];
        pjob jb; ptype ty; pops o;
        if (views(j, g, off, t, p, a, x, a2a, batch, speed, mem, bwi, bwe, gpn, hbm, &jb, &ty)) return -1;
        build_ops(&jb, &ty, f_ref, n_ops, n, &o);
        int smax = o.O < n ? o.O : n;
        /* every grid's proxy and price */
        double Tg[PO_MAX_OPS + 1][PO_MAX_M];
        pgrid G[PO_MAX_OPS + 1][PO_MAX_M];
        double Tmin = INFINITY;
        for (int s = 1; s <= smax; ++s) {
            grid_proxies(&jb, &ty, &o, kap, n, s, m_values, n_m, G[s]);
            for (int k = 0; k < n_m; ++k) {
                Tg[s][k] = G[s][k].ok ? G[s][k].T : INFINITY;
                if (Tg[s][k] < Tmin) Tmin = Tg[s][k];
            }
        }
        double* o4 = out + 4 * (int64_t)q;
        int32_t* pq = plan + 52 * (int64_t)q;
        for (int z = 0; z < 52; ++z) pq[z] = 0;
        if (!(Tmin < INFINITY)) {
            o4[0] = INFINITY; o4[1] = 0.0; o4[2] = 0.0; o4[3] = 0.0;
            continue;
        }
        double lim = Tmin * (1.0 + tie_eps);
        int bs = 0, bk = 0, done = 0;
        for (int s = 1; s <= smax && !done; ++s) {
            /* within a degree, the smaller B first: m_values ascending */
            int kbest = -1;
            for (int k = 0; k < n_m; ++k) {
                if (!(Tg[s][k] <= lim)) continue;
                if (kbest < 0 || m_values[k] < m_values[kbest]) kbest = k;
            }
            if (kbest >= 0) { bs = s; bk = kbest; done = 1; }
        }
        pgrid* w = &G[bs][bk];
        o4[0] = w->T; o4[1] = w->b2; o4[2] = w->lcomm; o4[3] = (double)jb.Bg / w->T;
        pq[0] = bs;
        pq[1] = m_values[bk];
        for (int z = 0; z <= bs; ++z) pq[2 + z] = w->pl.bound[z];
        for (int z = 0; z < bs; ++z) { pq[19 + z] = w->pl.Dn[z]; pq[35 + z] = w->pl.tp[z]; }
    }
    return 0;
}
