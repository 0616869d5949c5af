/*
 * arena.h - C ABI of the MI355X plan-space estimator.
 *
 * For every cell (job, GPU type, GPU count) the library enumerates the
 * adaptive-parallelism plans (dp, tp, pp, m) the cell admits, partitions the
 * job's profiled per-layer costs into pp contiguous stages so that the
 * slowest stage is as fast as possible, prices each plan with the 1F1B
 * pipeline model, and keeps the best plan.  The result is the job x grid
 * iteration-time and throughput matrix a cluster scheduler consumes.
 *
 * Paper: "Arena: Efficiently Training Large Models via Dynamic Scheduling
 * and Adaptive Parallelism Co-Design" (arXiv 2403.16125).
 *   - plan space: the joint scheduling x parallelism space, Eq. 1, sharded
 *     into grids of fixed resources and pipeline degree (Sec. 3.2);
 *   - balanced stages: at a fixed pipeline degree the plan with balanced
 *     inter-stage load wins because a pipeline runs at its slowest stage
 *     (Sec. 3.2);
 *   - stage latency = sum of its operators' latencies; comm latency is
 *     proportional to volume; end-to-end 1F1B latency = first microbatch
 *     through every stage + (B-1) microbatches of the slowest stage with p2p
 *     overlapped (Sec. 3.4);
 *   - intra-stage comm per microbatch and comm once per iteration (Eq. 4);
 *     intra-stage parallelism chosen within memory limits (Sec. 3.3);
 *   - the best grid per resource feeds the throughput matrix Thr[m,n]
 *     (Sec. 3.5, Eq. 5) and iteration times T[m,n] (Eq. 7).
 *
 * Model details the paper leaves open (units, memory model, link choice,
 * tie-breaks) are fixed as follows.  Units are SI: seconds, bytes, bytes/s.
 *   u_l    = t_l / (Bg speed tp)
 *            + kappa [tp>1] 8 (tp-1)/tp x_l / bw_intra      (TP all-reduces)
 *            + kappa [dp tp > 1] a2a_l / bw_inter           (MoE all-to-all)
 *   stage k holds layers [c_k, c_{k+1}); S_k = sum of u over it;
 *   b      = Bg / (dp m) samples per microbatch
 *   T      = sum_k (b S_k + p2p_k) + (m-1) b max_k S_k + max_k AR_k
 *   p2p_k  = kappa 2 b x_{c_{k+1}-1} / B_pp   (k < pp-1)
 *   AR_k   = kappa [dp>1] 2 (dp-1)/dp (P_k/tp) / B_dp
 *   Mem_k  = 4 P_k / tp + min(m, pp-k) b A_k / tp  <= mem   (feasibility)
 *   B_pp   = bw_intra if n <= gpus_per_node else bw_inter
 *   B_dp   = bw_intra if dp tp divides gpus_per_node else bw_inter
 *   cuts   = lexicographically smallest cut vector attaining min max_k S_k
 *   choice = smallest (pp, tp, m) among feasible plans with
 *            T <= T_min (1 + tie_eps).
 * Arithmetic is IEEE double; outputs are rounded to float.
 *
 * Conventions.  Every function returns an arena_status and never throws.
 * Arguments are validated on the host before anything is enqueued; on
 * error nothing is written and arena_last_error() says why.  A context is
 * used by one thread at a time and one stream at a time.  Device pointers
 * are caller-owned and must stay valid while bound.
 */
#ifndef ARENA_H
#define ARENA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum arena_status {
    ARENA_OK = 0,
    ARENA_ERR_INVALID_ARG = 1,   /* a null pointer, a size or value out of range */
    ARENA_ERR_OUT_OF_MEMORY = 2, /* a device or pinned host allocation failed */
    ARENA_ERR_DEVICE = 3,        /* a HIP call failed; the message carries HIP's string */
    ARENA_ERR_NOT_READY = 4,     /* a required bind/set call has not been made */
    ARENA_ERR_UNSUPPORTED = 5    /* valid input beyond the library's limits */
} arena_status;

/* Limits (ARENA_ERR_UNSUPPORTED beyond them). */
#define ARENA_MAX_LAYERS 128          /* layers (clustered operators) per job */
#define ARENA_MAX_GPU_COUNT 1024      /* GPUs of one cell */
#define ARENA_MAX_GPUS_PER_NODE 31    /* node size, bounds tp */
#define ARENA_MAX_M_VALUES 16         /* distinct microbatch counts */
#define ARENA_MAX_M 127               /* largest microbatch count */
#define ARENA_MAX_PLANS_PER_CELL 256  /* plans one cell may admit */
#define ARENA_MAX_TYPES 64
#define ARENA_MAX_COUNTS 512

/* Packed plan word: dp bits 0-10, tp bits 11-15, pp bits 16-23, m bits
 * 24-30, bit 31 set when the cell has a feasible plan.  An infeasible cell
 * has plan 0, t_iter +inf and thr 0. */
#define ARENA_PLAN_DP(w) ((uint32_t)(w) & 0x7FFu)
#define ARENA_PLAN_TP(w) (((uint32_t)(w) >> 11) & 0x1Fu)
#define ARENA_PLAN_PP(w) (((uint32_t)(w) >> 16) & 0xFFu)
#define ARENA_PLAN_M(w) (((uint32_t)(w) >> 24) & 0x7Fu)
#define ARENA_PLAN_FEASIBLE(w) (((uint32_t)(w) >> 31) & 1u)

typedef struct arena_ctx arena_ctx;

/* Profiled jobs (the planner's per-operator inputs, Sec. 3.4).  Layers of
 * job j are [layer_offset[j], layer_offset[j+1]). */
typedef struct arena_jobs_desc {
    int32_t n_jobs;
    int32_t n_layers_total;
    const int32_t* layer_offset; /* HOST, n_jobs+1, copied; offset[0]=0, increasing */
    const int32_t* batch;        /* HOST, n_jobs, copied; global batch size >= 1 */
    const float* t;   /* DEVICE, fwd+bwd seconds of the layer for the whole global
                         batch on one GPU of speed 1 */
    const float* p;   /* DEVICE, parameter bytes */
    const float* a;   /* DEVICE, stored activation bytes per sample */
    const float* x;   /* DEVICE, output activation bytes per sample */
    const float* a2a; /* DEVICE, all-to-all bytes per sample, 0 on dense layers */
} arena_jobs_desc;

/* GPU types and the GPU counts of the grid (the scheduling plans (n, type)
 * of Sec. 3.2).  All arrays are host arrays and are copied. */
typedef struct arena_grids_desc {
    int32_t n_types;
    const float* speed;           /* relative to the speed-1 GPU the times refer to, > 0 */
    const float* mem_bytes;       /* per GPU, > 0 */
    const float* bw_intra;        /* bytes/s inside a node, > 0 (+inf allowed) */
    const float* bw_inter;        /* bytes/s across nodes, > 0 (+inf allowed) */
    const int32_t* gpus_per_node; /* 1..ARENA_MAX_GPUS_PER_NODE */
    int32_t n_counts;
    const int32_t* counts;        /* 1..ARENA_MAX_GPU_COUNT, distinct */
} arena_grids_desc;

/* Work of the last arena_estimate (device-side tallies; plans_skipped is the
 * plan space less the plans priced). */
typedef struct arena_counters {
    int64_t cells;            /* cells written */
    int64_t plans;            /* plans priced */
    int64_t problems;         /* stage-partition problems solved */
    int64_t dp_entries;       /* partition-recursion entries evaluated */
    int64_t infeasible_cells; /* cells with no feasible plan */
    int64_t plans_skipped;    /* plans never priced: a lower bound of their iteration time
                                 lies above the tie window of a plan already priced, or no
                                 stage split of their degree fits memory.
                                 plans + plans_skipped = the plan space */
    int64_t alg_ops;          /* algorithmic operations of the work done: 8 per layer of each
                                 solved problem (layer costs and prefix), 8 per recursion entry,
                                 4 L per priced pipeline degree (cuts), 12 pp + 40 per priced
                                 plan; under ARENA_PARTITION_MEMORY also 4 L per memory-only
                                 split test and per memory-rule cut vector */
    int64_t mem_partitions;   /* memory-rule partitions solved (ARENA_PARTITION_MEMORY) */
} arena_counters;

/* Exact size of the plan space of the bound tables (host-side count). */
typedef struct arena_space_size {
    int64_t cells;
    int64_t plans;
    int32_t max_plans_per_cell;
    int32_t max_layers;
} arena_space_size;

/* Create a context for HIP device `hip_device`.  Allocates nothing on the
 * device and makes no HIP call; device state is created lazily. */
arena_status arena_create(int hip_device, arena_ctx** out);

/* Free the context and everything it allocated.  NULL is allowed.  The
 * caller synchronises streams that still use the context first. */
void arena_destroy(arena_ctx* ctx);

/* Text of the last error on ctx (empty when none).  Owned by ctx, valid until
 * the next call on ctx.  NULL ctx gives a static string. */
const char* arena_last_error(const arena_ctx* ctx);

/* Name of a status code (static string). */
const char* arena_status_string(arena_status s);

/* Bind jobs.  Validates the host arrays, then checks on the device that every
 * per-layer value is finite and >= 0 (synchronous; INVALID_ARG otherwise) and
 * records which jobs have all-to-all layers.  Keeps the device pointers. */
arena_status arena_bind_jobs(arena_ctx* ctx, const arena_jobs_desc* jobs);

/* Bind GPU types and counts (host-only, copied).  Resets kappa to 1. */
arena_status arena_bind_grids(arena_ctx* ctx, const arena_grids_desc* grids);

/* Per-grid contention factor kappa[type * n_counts + count_index] (finite,
 * > 0), multiplying every communication term.  Host array, copied; uploaded
 * by the next arena_estimate on its stream.  n = n_types * n_counts. */
arena_status arena_set_kappa(arena_ctx* ctx, const float* kappa_host, int32_t n);

/* Microbatch counts to consider (distinct, 1..ARENA_MAX_M) and the relative
 * tie tolerance of the per-cell choice (0 <= tie_eps < 1e-2). */
arena_status arena_set_plan_space(arena_ctx* ctx, const int32_t* m_values, int32_t n_m,
                                  double tie_eps);

/* Bound pruning of the plan search (default: on).  With it, a pipeline
 * degree whose lower bound of the iteration time lies above the tie window of
 * a plan already priced, or none of whose stage splits fits memory, is not
 * priced, and the partition recursion stops after the last degree still
 * wanted.  The results are identical either way; only the work differs (see
 * plans_skipped).  0 turns it off, any other value on. */
arena_status arena_set_bound_pruning(arena_ctx* ctx, int32_t enabled);

/* Partition rules (arena_set_partition_rule). */
#define ARENA_PARTITION_BALANCED 0
#define ARENA_PARTITION_MEMORY 1
#define ARENA_PARTITION_EXACT_T 2
#define ARENA_EXACT_T_MAX_LAYERS 96   /* layers per job under ARENA_PARTITION_EXACT_T */

/* Which stage partition prices a plan (default ARENA_PARTITION_BALANCED).
 *   BALANCED  the canonical balanced partition (Sec. 3.2: a pipeline runs at
 *             its slowest stage, so the stages minimise the largest stage
 *             cost), then the memory check; a plan whose balanced stages do
 *             not fit is infeasible.
 *   MEMORY    the same criterion over the splits whose every stage fits
 *             memory (Sec. 3.3 picks parallelism within memory limits):
 *             stage k of pp holds 4 P_k/tp + min(m, pp-k) b A_k/tp bytes, at
 *             most mem; the lexicographically smallest such split of least
 *             largest stage cost.  A plan is infeasible only when no split
 *             fits.  Plans whose balanced split fits are priced as under
 *             BALANCED, so no cell gets slower; cut rows follow the rule.
 *   EXACT_T   the split of least iteration time: the whole 1F1B time of Sec.
 *             3.4 (with Eq. 4's all-reduce) among the splits whose every
 *             stage fits memory (the MEMORY rule's test, a stage's bytes as
 *             differences of running totals).  The stage costs summed over
 *             the stages do not depend on the split, so it minimises
 *             Phi = ((m-1) b Smax + cX X) + cP Pmax, evaluated in that order:
 *             Smax the slowest stage per sample, X = x_{c_1-1} + (x_{c_2-1} +
 *             ...) the boundary bytes added from the back, Pmax the largest
 *             stage's parameter bytes, cX = kappa 2 b / B_pp, cP = kappa 2
 *             (dp-1)/dp / (tp B_dp) (0 when dp = 1).  Ties: the least (Phi,
 *             Smax, Pmax, X), then the lexicographically smallest cuts.  No
 *             cell is slower than under MEMORY, and the cell's best time
 *             never grows with a link bandwidth.  t_iter = b U_L + Phi.
 *             Jobs of at most ARENA_EXACT_T_MAX_LAYERS layers (the exact
 *             method visits pairs of thresholds, each a recursion over
 *             stages); arena_estimate returns UNSUPPORTED beyond, and with
 *             comm tables.
 * Takes effect at the next arena_estimate; INVALID_ARG for other values. */
arena_status arena_set_partition_rule(arena_ctx* ctx, int32_t rule);

#define ARENA_MAX_COMM_POINTS 16   /* samples per communication latency table */

/* Communication latency interpolated in profiled tables instead of volume /
 * bandwidth.  The paper profiles each communication primitive offline at
 * sampled volumes on the target interconnect and, online, interpolates its
 * latency by volume under the same primitive and topology (Sec. 3.4).  Here
 * each GPU type has one table per link -- link 0 inside a node, link 1
 * across nodes -- of n_points samples: volumes[(g*2 + link)*n_points + k]
 * bytes (the first 0, strictly increasing, finite) with latencies[...]
 * seconds (finite, >= 0, non-decreasing).  f(v) = 0 when nothing moves, else
 * linear between the samples around v, extended by the first or last
 * segment.  With tables set, every communication term takes its latency
 * from its link's table, scaled by kappa:
 *   tensor-parallel   4 f_intra(2 (tp-1)/tp b x_l)  per layer and microbatch
 *   MoE all-to-all    f_inter(b a2a_l)              per layer and microbatch, dp tp > 1
 *   p2p               2 f_pp(b x_last)              per stage boundary (fill term)
 *   DP all-reduce     f_dp(2 (dp-1)/dp P_k/tp)      per iteration, dp > 1
 * (b = Bg/(dp m); f_pp, f_dp on the links of the balanced model), and the
 * stage costs are per microbatch: each plan (dp, tp, pp, m) gets the
 * canonical balanced partition of its own per-microbatch layer costs (with
 * bound pruning, a plan whose lower bound lies past the tie window of a plan
 * already priced is skipped; the results are the same), and the per-cell choice,
 * outputs and cut rows are as without tables.  Tables linear through the
 * origin reproduce the volume / bandwidth model.  Host arrays, copied;
 * uploaded by the next arena_estimate.  Needs grids bound (the tables follow
 * their type count; rebinding grids with another type count makes
 * arena_estimate return NOT_READY until tables are set again).  n_points = 0
 * returns to volume / bandwidth.  With tables, arena_estimate returns
 * UNSUPPORTED under ARENA_PARTITION_MEMORY.  INVALID_ARG on bad values,
 * nothing kept. */
arena_status arena_set_comm_tables(arena_ctx* ctx, int32_t n_points, const double* volumes,
                                   const double* latencies);

/* Size of the plan space of the bound tables (host computation, no HIP
 * call).  Needs jobs, grids and plan space bound. */
arena_status arena_space_size_get(const arena_ctx* ctx, arena_space_size* out);

/* Estimate every cell, asynchronously on `stream` (a hipStream_t; NULL is the
 * null stream).  Outputs are caller-owned DEVICE arrays of n_jobs * n_types *
 * n_counts entries, cell (j, g, c) at index (j * n_types + g) * n_counts + c:
 *   t_iter  float   iteration time of the best plan (s), +inf if none fits
 *   thr     float   throughput Bg / t_iter (samples/s), 0 if none fits
 *   plan    uint32  packed plan word (see ARENA_PLAN_*)
 *   cuts    uint8   nullable; row of cuts_stride bytes per cell holding the
 *                   first layer of stages 1..pp-1, then 0xFF.
 *                   cuts_stride >= max layers - 1 when cuts is not NULL. */
arena_status arena_estimate(arena_ctx* ctx, float* t_iter, float* thr, uint32_t* plan,
                            uint8_t* cuts, int32_t cuts_stride, void* stream);

/* Cap on the device memory the library allocates for this context: its
 * copies of the job offsets, batches, grid tables and contention factors,
 * the work order, the tallies, the communication tables and the estimate
 * blocks' caches of pure-compute splits (the caller's arrays are not
 * counted).  bytes = 0 (the default) sets no cap.  An arena_estimate whose
 * bound workload needs more returns ARENA_ERR_OUT_OF_MEMORY before anything
 * is allocated, enqueued or written (the need is 4 (J+1) + 4 J + 40 T + 8 NC
 * + 4 T NC + 4 J T bytes plus the communication tables and about 2 KB, for J
 * jobs, T types and NC counts, plus 8448 bytes per estimate block: one block
 * per item up to four per compute unit, 8.3 MiB on 256 CUs).  The tables are
 * checked first, before the device is asked for its CU count.  INVALID_ARG
 * for a negative value.  arena_estimate also returns OUT_OF_MEMORY when a
 * device allocation fails. */
arena_status arena_set_workspace_limit(arena_ctx* ctx, int64_t bytes);

#define ARENA_NOALLOC_SCRATCH_BYTES (16u << 20)

/* arena_estimate for callers that cannot allocate device memory (work under
 * stream capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, arguments, outputs and errors, but every
 * library-owned device buffer of the call (job offsets and batches, grid
 * tables, contention factors, work order, tallies, communication tables,
 * the blocks' split caches) is placed in one statically sized device array
 * of ARENA_NOALLOC_SCRATCH_BYTES per GPU, which the library holds until the process ends; the call makes no
 * device or pinned allocation (it copies the tables from the context's host
 * copies into the array on `stream` each time, and on the first call for
 * a set of job tables runs the value check, which synchronises the stream).
 * Every call on one GPU shares that GPU's array and leaves its contents
 * (the tallies of the last call, which arena_get_counters reads): calls that
 * overlap on one GPU, from any context or stream, race and must be ordered by
 * the caller.  Returns ARENA_ERR_OUT_OF_MEMORY, with nothing enqueued or
 * written, when the bound workload needs more than the array (about
 * 4 J T + 8 J + 4 T NC bytes of tables plus 8448 bytes per estimate block,
 * four per compute unit; for example 16384 jobs x 8 types x 131 counts need
 * 0.7 MB of tables and 8.3 MiB of caches on 256 CUs). */
arena_status arena_estimate_noalloc(arena_ctx* ctx, float* t_iter, float* thr, uint32_t* plan,
                                    uint8_t* cuts, int32_t cuts_stride, void* stream);

/* Tallies of the last arena_estimate or arena_estimate_noalloc.
 * Synchronises the device. */
arena_status arena_get_counters(arena_ctx* ctx, arena_counters* out);

/* ------------------------------------------------------------------ */
/* Proxy-plan planner                                                   */
/* ------------------------------------------------------------------ */

#define ARENA_MAX_PROXY_OPS 16

/* The load-aware planner of Sec. 3.3, which picks one plan per grid without
 * execution, for every cell of the bound jobs and grids (same bindings,
 * plan space, contention factors and cell order as arena_estimate):
 *   - the job's L layers form O = min(L, n_ops) clustered operators,
 *     operator i holding layers floor(iL/O) .. floor((i+1)L/O) - 1;
 *   - an operator's load is its roofline time (Eq. 2): FLOPs = f_ref * sum t
 *     over its layers, memory traffic = sum (p + batch a); load =
 *     max(FLOPs / (speed f_ref), traffic / hbm_bw) -- FLOPs over the rate
 *     the roofline allows at the operator's arithmetic intensity;
 *   - its GPU share is proportional: d_i = (load_i / sum load) n;
 *   - for every pipeline degree s (one grid per s, Sec. 3.2) every
 *     contiguous grouping of the operators into s stages gets power-of-two
 *     stage GPU counts summing to n that minimise the computation bias of
 *     Eq. 3 (the sorted pairing of each multiset; the bias summed over
 *     stages in stage order; ties: the lexicographically larger sorted
 *     multiset, equal shares give the larger count to the earlier stage);
 *   - for each microbatch count B of the plan space, among groupings whose
 *     every stage fits memory, the proxy plan has the least bias, then the
 *     least communication load of Eq. 4, (B-1) max_j C_j + sum_j C_j +
 *     sum_j AR_j, with each stage's (dp, tp) chosen for the least
 *     communication per iteration within memory (ties: smaller tp), then the
 *     lexicographically smallest cut vector;
 *   - each grid's proxy is priced by the 1F1B model of arena_estimate with
 *     per-stage GPU counts (samples per replica Bg / (dp_j B); point-to-point
 *     traffic Bg / (B min(dp_j, dp_j+1)) samples per boundary); the cell
 *     keeps the fastest grid, T within (1 + tie_eps) of the least counting as
 *     a tie, broken by fewer stages, then fewer microbatches.
 * Outputs (caller-owned device buffers, C cells in arena_estimate's order):
 *   t_iter  f32 [C]  iteration time of the chosen proxy plan (+inf: no grid fits)
 *   thr     f32 [C]  batch / t_iter (0 when infeasible)
 *   plan    u64 [3C] word 0: bits 0-14 stage starts (bit i-1 set: a stage
 *                    starts at operator i), bits 16-20 s, bits 24-30 B, bit
 *                    31 feasible; word 1: log2 of each stage's GPU count,
 *                    4 bits per stage (stage j at bits 4j); word 2: log2 of
 *                    each stage's tensor degree, same layout.  All zero when
 *                    infeasible.
 * Asynchronous on `stream`.  A job whose operators all have zero load has no
 * proxy plan.  Host checks (jobs, grids and plan space bound; hbm_bw, f_ref
 * and n_ops in range; output pointers; at most 2^31 - 1 cells; at most 1280
 * power-of-two splits of one count into one stage count) return an error
 * before anything is enqueued. */
typedef struct arena_proxy_desc {
    const float* hbm_bw;   /* HOST [n_types] memory bandwidth of each type, bytes/s, finite > 0; copied */
    double f_ref;          /* FLOP/s of a speed-1.0 GPU, finite > 0 */
    int32_t n_ops;         /* operators per job (clusters of consecutive layers), 1..ARENA_MAX_PROXY_OPS */
} arena_proxy_desc;

arena_status arena_proxy_estimate(arena_ctx* ctx, const arena_proxy_desc* d, float* t_iter, float* thr,
                                  uint64_t* plan, void* stream);

/* ------------------------------------------------------------------ */
/* Scheduler consumer of the throughput matrix                          */
/* ------------------------------------------------------------------ */

#define ARENA_MAX_SCHED_JOBS 65536
#define ARENA_MAX_SCHED_DEPTH 256
#define ARENA_MAX_SCHED_CAPACITY (1 << 24)   /* GPUs of one type */

/* Scheduling objectives (arena_sched_desc.objective). */
#define ARENA_SCHED_THROUGHPUT 0   /* Eq. 5: maximise the summed throughput */
#define ARENA_SCHED_FAIRNESS 1     /* Eq. 7: minimise the largest finish-time-fairness ratio */

/* One scheduling step over a throughput matrix (for instance the thr output
 * of arena_estimate): event-driven scheduling with the throughput objective
 * (Sec. 3.5, Algorithm 1, Eq. 5).  Queued jobs are visited in queue order;
 * each launches on its fastest grid that fits the free GPUs (ties: fewer
 * GPUs, then the lower type), or, while it does not fit and fewer than
 * `depth` moves were made, the running job whose scale-down to its next
 * smaller count with throughput > 0 loses the least throughput per freed GPU
 * (on a type the queued job can use; ties: lower job id) is scaled down;
 * moves of a job that still does not fit are undone.  A job that does not
 * launch stops the visit if its priority class is above the smallest class
 * that failed before it.  Finally up to `depth` scale-ups are made, each the
 * running job's move to a larger count on its type, within the free GPUs,
 * with the largest throughput gained per added GPU (ties: smaller count,
 * lower job id).  Costs and gains are float64 from the float32 matrix.
 * Running jobs keep their GPU type.  Asynchronous on `stream`; everything runs
 * in one workgroup of the device. */
typedef struct arena_sched_desc {
    int32_t n_jobs, n_types, n_counts;
    const float* thr;            /* DEVICE [n_jobs * n_types * n_counts], (j, g, c) at (j*T + g)*NC + c;
                                    samples/s, finite and >= 0, 0 where the grid does not fit (other
                                    values are not checked: the decisions are then unspecified) */
    const int32_t* counts;       /* HOST [n_counts], strictly ascending, 1..ARENA_MAX_GPU_COUNT; copied */
    const int32_t* capacity;     /* HOST [n_types], GPUs of each type, 0..ARENA_MAX_SCHED_CAPACITY; copied */
    int32_t* alloc_type;         /* DEVICE [n_jobs] in/out: a running job's type, -1 if not running */
    int32_t* alloc_count;        /* DEVICE [n_jobs] in/out: a running job's count index */
    const int32_t* queue;        /* DEVICE [n_queue]: queued job ids (distinct, not running), visiting order */
    const int32_t* priority;     /* DEVICE [n_queue]: priority class of each queued job, >= 0 */
    int32_t n_queue;             /* 0..n_jobs */
    int32_t depth;               /* search depth D, 1..ARENA_MAX_SCHED_DEPTH */
    int32_t* launched;           /* DEVICE [n_queue] out: 1 if the job launched */
    int32_t* result;             /* DEVICE [8] out: status (0 ok; 1 the running jobs exceed the
                                    capacity; 2 an index out of range, a queued job running or listed
                                    twice, a negative class or a bad deadline value -- nothing is
                                    changed then), scale-downs kept, launches, scale-ups, decisions
                                    taken (launch, scale-down and scale-up searches), candidates they
                                    examined (64-bit: low word, high word), 0 */
    /* Deadline constraint (Eq. 6), optional: all three NULL to schedule without it.  With it, a grid
     * is open to job i only if batch_i iters_i / thr <= deadline_i (fp64): launches, scale-downs (the
     * largest smaller count still meeting it) and scale-ups (a larger count meeting it) consider open
     * grids only, and the usable types of a queued job are those with an open grid. */
    const int32_t* batch;        /* DEVICE [n_jobs] global batch size, > 0 */
    const float* iters;          /* DEVICE [n_jobs] remaining iterations, finite >= 0 */
    const float* deadline;       /* DEVICE [n_jobs] seconds left to the deadline, > 0 (+inf: none) */
    /* Objective: ARENA_SCHED_THROUGHPUT (the searches above) or ARENA_SCHED_FAIRNESS (Eq. 7, which
     * needs batch and iters; deadline may then be NULL).  Under fairness a job at throughput thr on n
     * GPUs has rho = batch iters / (thr n) (fp64; the grid's GPU count is the resource measure Q), and
     * the searches rank by it: a scale-down moves the job whose rho after the step is least (ties:
     * lower job id); a scale-up takes each running job's larger count within the free GPUs (and open,
     * with deadlines) of least rho (ties: smaller count), if below its current rho, and moves the job
     * whose current rho is largest (ties: lower job id).  Launches are as above. */
    int32_t objective;
} arena_sched_desc;

/* Host checks (sizes, pointers, counts, capacity, depth) return an error
 * before anything is enqueued; device-side state errors are reported in
 * result[0].  n_jobs <= ARENA_MAX_SCHED_JOBS, n_types <= ARENA_MAX_TYPES,
 * n_counts <= ARENA_MAX_COUNTS. */
arena_status arena_schedule(arena_ctx* ctx, const arena_sched_desc* d, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ARENA_H */
