// Host side of the C ABI declared in include/arena.h: argument validation,
// context state, lazy device set-up, table uploads and kernel launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <map>
#include <numeric>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "arena.h"
#include "arena_internal.h"

using arena::TypeDev;

static_assert(ARENA_NOALLOC_SCRATCH_BYTES == arena::kNoallocScratchBytes, "scratch size of the header and the kernels");
static_assert(ARENA_EXACT_T_MAX_LAYERS == arena::kExactTMaxLayers, "exact-T layer limit of the header and the kernels");

struct arena_ctx {
    int device = 0;
    std::string err;

    // jobs (host copies of per-job scalars; device pointers are the caller's)
    bool jobs_bound = false;
    bool jobs_checked = false;     // device-side value check done for this bind
    int32_t n_jobs = 0, n_layers = 0, max_layers = 0;
    std::vector<int32_t> off, batch;
    const float *t = nullptr, *p = nullptr, *a = nullptr, *x = nullptr, *q = nullptr;
    bool jobs_dirty = true;

    // grids
    bool grids_bound = false;
    int32_t n_types = 0, n_counts = 0;
    std::vector<TypeDev> types;
    std::vector<int32_t> counts;
    std::vector<float> kappa;
    bool grids_dirty = true, kappa_dirty = true;

    // plan space
    bool space_set = false;
    std::vector<int32_t> m_values;
    double tie_eps = 1e-6;
    bool prune = true;
    int32_t partition_rule = ARENA_PARTITION_BALANCED;

    // interpolated communication latency: volumes then latencies, [T][2][K]
    int32_t tab_k = 0, tab_types = 0;
    std::vector<double> tab;
    bool tab_dirty = false;
    double* d_tab = nullptr;
    size_t cap_tab = 0;

    // cached space size
    bool size_valid = false;
    arena_space_size size{};

    // device state
    bool dev_ready = false;
    int32_t* d_off = nullptr;
    int32_t* d_batch = nullptr;
    size_t cap_jobs = 0, cap_batch = 0;
    TypeDev* d_types = nullptr;
    int32_t* d_counts = nullptr;
    float* d_kappa = nullptr;
    size_t cap_types = 0, cap_counts = 0, cap_kappa = 0;
    int32_t* d_item_order = nullptr;
    int32_t* d_count_order = nullptr;
    size_t cap_items = 0, cap_corder = 0;
    bool order_dirty = true;
    bool horder_valid = false;                  // host copies of the work order below are current
    std::vector<int32_t> h_iorder, h_corder;
    int32_t h_qoff[arena::kQueues + 1] = {};    // queue q's items: h_iorder[h_qoff[q] .. h_qoff[q+1])
    int64_t ws_limit = 0;                       // cap on library-owned device bytes, 0: none
    unsigned long long* d_counters = nullptr;
    const unsigned long long* last_counters = nullptr;   // tallies of the last estimate
    int64_t last_space_plans = 0;               // the plan space of the last estimate
    unsigned long long* h_counters = nullptr;   // pinned
    unsigned long long* d_queue = nullptr;      // the estimate and proxy kernels' item queue
    uint8_t* d_pcut = nullptr;                  // the estimate blocks' caches of pure-compute splits
    size_t cap_pcut = 0;
    int n_cus = 0;
    float* h_kappa[2] = {nullptr, nullptr};     // pinned staging, double-buffered
    hipEvent_t kappa_done[2] = {nullptr, nullptr};
    size_t cap_hkappa = 0;
    int kslot = 0;

    // proxy planner: power-of-two multisets per (count, stage count), memory bandwidths
    bool msets_dirty = true;
    std::vector<unsigned long long> msets;
    std::vector<int32_t> mset_off;
    unsigned long long* d_msets = nullptr;
    int32_t* d_mset_off = nullptr;
    double* d_hbm = nullptr;
    size_t cap_msets = 0, cap_mset_off = 0, cap_hbm = 0;

    // scheduler: device copy of counts and capacity, staged through pinned memory
    int32_t* d_sched = nullptr;
    int32_t* h_sched = nullptr;
    size_t cap_sched = 0, cap_hsched = 0;
    hipEvent_t sched_done = nullptr;
};

namespace {

arena_status fail(arena_ctx* c, arena_status s, const char* fmt, ...)
{
    if (c) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof(buf), fmt, ap);
        va_end(ap);
        c->err = buf;
    }
    return s;
}

arena_status hip_fail(arena_ctx* c, hipError_t e, const char* what)
{
    return fail(c, ARENA_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool is_pos_finite_or_inf(float v) { return v > 0.0f && !std::isnan(v); }

// Plans of one cell: tp | n, tp | node size, pp | n/tp, pp <= L, dp = n/(tp pp),
// m listed with dp*m | Bg.
int64_t plans_of_cell(int n, int gpn, int L, int Bg, const std::vector<int32_t>& ms)
{
    int64_t cnt = 0;
    for (int tp = 1; tp <= n && tp <= gpn; ++tp) {
        if (n % tp || gpn % tp) continue;
        const int q = n / tp;
        for (int pp = 1; pp <= q && pp <= L; ++pp) {
            if (q % pp) continue;
            const int dp = q / pp;
            for (int m : ms)
                if (Bg % (dp * m) == 0) ++cnt;
        }
    }
    return cnt;
}

void free_device(arena_ctx* c)
{
    (void)hipFree(c->d_off);
    (void)hipFree(c->d_batch);
    (void)hipFree(c->d_types);
    (void)hipFree(c->d_counts);
    (void)hipFree(c->d_kappa);
    (void)hipFree(c->d_item_order);
    (void)hipFree(c->d_count_order);
    (void)hipFree(c->d_counters);
    (void)hipHostFree(c->h_counters);
    (void)hipFree(c->d_queue);
    c->d_queue = nullptr;
    (void)hipFree(c->d_pcut);
    c->d_pcut = nullptr;
    c->cap_pcut = 0;
    (void)hipFree(c->d_msets);
    (void)hipFree(c->d_mset_off);
    (void)hipFree(c->d_hbm);
    (void)hipFree(c->d_tab);
    c->d_tab = nullptr;
    c->cap_tab = 0;
    c->tab_dirty = c->tab_k > 0;
    c->d_msets = nullptr;
    c->d_mset_off = nullptr;
    c->d_hbm = nullptr;
    c->cap_msets = c->cap_mset_off = c->cap_hbm = 0;
    c->msets_dirty = true;
    (void)hipFree(c->d_sched);
    (void)hipHostFree(c->h_sched);
    if (c->sched_done) (void)hipEventDestroy(c->sched_done);
    c->d_sched = c->h_sched = nullptr;
    c->cap_sched = c->cap_hsched = 0;
    c->sched_done = nullptr;
    for (int i = 0; i < 2; ++i) {
        (void)hipHostFree(c->h_kappa[i]);
        if (c->kappa_done[i]) (void)hipEventDestroy(c->kappa_done[i]);
    }
    c->d_off = c->d_batch = nullptr;
    c->d_types = nullptr;
    c->d_counts = nullptr;
    c->d_kappa = nullptr;
    c->d_item_order = nullptr;
    c->d_count_order = nullptr;
    c->d_counters = nullptr;
    c->h_counters = nullptr;
    c->h_kappa[0] = c->h_kappa[1] = nullptr;
    c->kappa_done[0] = c->kappa_done[1] = nullptr;
}

// Selects ctx->device for the duration of a call, restoring the caller's.
struct DeviceGuard {
    int prev = -1;
    hipError_t status = hipSuccess;
    explicit DeviceGuard(int dev)
    {
        status = hipGetDevice(&prev);
        if (status == hipSuccess && prev != dev) status = hipSetDevice(dev);
        else if (status == hipSuccess) prev = -1;
    }
    ~DeviceGuard()
    {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

template <typename T>
hipError_t ensure_capacity(T** ptr, size_t* cap, size_t n)
{
    if (*cap >= n && *ptr) return hipSuccess;
    (void)hipFree(*ptr);
    *ptr = nullptr;
    *cap = 0;
    hipError_t e = hipMalloc((void**)ptr, sizeof(T) * (n ? n : 1));
    if (e == hipSuccess) *cap = n;
    return e;
}

arena_status ensure_device(arena_ctx* c, hipStream_t stream)
{
    hipError_t e;
    if (!c->dev_ready) {
        if ((e = hipMalloc((void**)&c->d_counters, sizeof(unsigned long long) * arena::kNumCounters)))
            return e == hipErrorOutOfMemory ? fail(c, ARENA_ERR_OUT_OF_MEMORY, "counters") : hip_fail(c, e, "hipMalloc");
        if ((e = hipHostMalloc((void**)&c->h_counters, sizeof(unsigned long long) * arena::kNumCounters, 0)))
            return hip_fail(c, e, "hipHostMalloc");
        if ((e = hipMalloc((void**)&c->d_queue, sizeof(unsigned long long) * arena::kQueues)))
            return e == hipErrorOutOfMemory ? fail(c, ARENA_ERR_OUT_OF_MEMORY, "queue") : hip_fail(c, e, "hipMalloc");
        if ((e = hipDeviceGetAttribute(&c->n_cus, hipDeviceAttributeMultiprocessorCount, c->device)))
            return hip_fail(c, e, "hipDeviceGetAttribute");
        for (int i = 0; i < 2; ++i)
            if ((e = hipEventCreateWithFlags(&c->kappa_done[i], hipEventDisableTiming)))
                return hip_fail(c, e, "hipEventCreate");
        c->dev_ready = true;
    }
    if (c->jobs_dirty) {
        if ((e = ensure_capacity(&c->d_off, &c->cap_jobs, (size_t)c->n_jobs + 1)))
            return fail(c, ARENA_ERR_OUT_OF_MEMORY, "job tables: %s", hipGetErrorString(e));
        if ((e = ensure_capacity(&c->d_batch, &c->cap_batch, (size_t)c->n_jobs)))
            return fail(c, ARENA_ERR_OUT_OF_MEMORY, "job tables: %s", hipGetErrorString(e));
        if ((e = hipMemcpyAsync(c->d_off, c->off.data(), sizeof(int32_t) * (c->n_jobs + 1),
                                hipMemcpyHostToDevice, stream)) ||
            (e = hipMemcpyAsync(c->d_batch, c->batch.data(), sizeof(int32_t) * c->n_jobs,
                                hipMemcpyHostToDevice, stream)) ||
            (e = hipStreamSynchronize(stream)))
            return hip_fail(c, e, "job table upload");
        c->jobs_dirty = false;
    }
    if (!c->jobs_checked) {
        arena::ValidateArgs v;
        v.layer_offset = c->d_off;
        v.n_jobs = c->n_jobs;
        v.arrays[0] = c->t; v.arrays[1] = c->p; v.arrays[2] = c->a; v.arrays[3] = c->x; v.arrays[4] = c->q;
        v.bad = c->d_counters;
        if ((e = arena::launch_zero_counters(c->d_counters, 1, stream)) ||
            (e = arena::launch_validate(v, stream)) ||
            (e = hipMemcpyAsync(c->h_counters, c->d_counters, sizeof(unsigned long long),
                                hipMemcpyDeviceToHost, stream)) ||
            (e = hipStreamSynchronize(stream)))
            return hip_fail(c, e, "job value check");
        if (c->h_counters[0] != 0)
            return fail(c, ARENA_ERR_INVALID_ARG,
                        "jobs: %llu per-layer values are negative or not finite",
                        (unsigned long long)c->h_counters[0]);
        c->jobs_checked = true;
    }
    if (c->grids_dirty) {
        size_t nk = (size_t)c->n_types * c->n_counts;
        if ((e = ensure_capacity(&c->d_types, &c->cap_types, (size_t)c->n_types)) ||
            (e = ensure_capacity(&c->d_counts, &c->cap_counts, (size_t)c->n_counts)) ||
            (e = ensure_capacity(&c->d_kappa, &c->cap_kappa, nk)))
            return fail(c, ARENA_ERR_OUT_OF_MEMORY, "grid tables: %s", hipGetErrorString(e));
        if ((e = hipMemcpyAsync(c->d_types, c->types.data(), sizeof(TypeDev) * c->n_types,
                                hipMemcpyHostToDevice, stream)) ||
            (e = hipMemcpyAsync(c->d_counts, c->counts.data(), sizeof(int32_t) * c->n_counts,
                                hipMemcpyHostToDevice, stream)) ||
            (e = hipStreamSynchronize(stream)))
            return hip_fail(c, e, "grid table upload");
        if (c->cap_hkappa < nk) {
            for (int i = 0; i < 2; ++i) {
                if (c->kappa_done[i]) (void)hipEventSynchronize(c->kappa_done[i]);
                (void)hipHostFree(c->h_kappa[i]);
                c->h_kappa[i] = nullptr;
                if ((e = hipHostMalloc((void**)&c->h_kappa[i], sizeof(float) * nk, 0)))
                    return fail(c, ARENA_ERR_OUT_OF_MEMORY, "pinned kappa staging");
            }
            c->cap_hkappa = nk;
        }
        c->grids_dirty = false;
        c->kappa_dirty = true;
    }
    if (c->kappa_dirty) {
        // stage into a pinned slot whose previous copy has completed, then copy
        // asynchronously on the caller's stream
        const size_t nk = (size_t)c->n_types * c->n_counts;
        const int s = c->kslot;
        if ((e = hipEventSynchronize(c->kappa_done[s]))) return hip_fail(c, e, "kappa slot wait");
        std::memcpy(c->h_kappa[s], c->kappa.data(), sizeof(float) * nk);
        if ((e = hipMemcpyAsync(c->d_kappa, c->h_kappa[s], sizeof(float) * nk,
                                hipMemcpyHostToDevice, stream)) ||
            (e = hipEventRecord(c->kappa_done[s], stream)))
            return hip_fail(c, e, "kappa upload");
        c->kslot ^= 1;
        c->kappa_dirty = false;
    }
    return ARENA_OK;
}

// Work order: jobs are dealt to the kernels' kQueues item queues (one per
// XCD) heaviest first, each to the queue with the least work so far; a queue
// lists its jobs heaviest first (so the longest items do not form the tail)
// with the (job, type) items of one job adjacent, heaviest type first, and
// within an item the largest GPU counts come first.  The estimate of work is
// plans x layers per cell.  Host copies, rebuilt when the bindings change.
void compute_orders(arena_ctx* c)
{
    if (c->horder_valid) return;
    std::vector<int32_t>& corder = c->h_corder;
    corder.resize((size_t)c->n_counts);
    std::iota(corder.begin(), corder.end(), 0);
    std::stable_sort(corder.begin(), corder.end(),
                     [&](int a, int b) { return c->counts[a] > c->counts[b]; });
    std::map<std::pair<int, int>, std::vector<double>> cost;
    const size_t items = (size_t)c->n_jobs * c->n_types;
    std::vector<double> icost(items);
    for (int j = 0; j < c->n_jobs; ++j) {
        const int L = c->off[j + 1] - c->off[j];
        auto key = std::make_pair(L, (int)c->batch[j]);
        auto it = cost.find(key);
        if (it == cost.end()) {
            std::vector<double> per((size_t)c->n_types, 0.0);
            for (int g = 0; g < c->n_types; ++g)
                for (int ci = 0; ci < c->n_counts; ++ci)
                    per[g] += (double)plans_of_cell(c->counts[ci], c->types[g].gpn, L, key.second,
                                                    c->m_values) * (double)(L + 16);
            it = cost.emplace(key, std::move(per)).first;
        }
        for (int g = 0; g < c->n_types; ++g) icost[(size_t)j * c->n_types + g] = it->second[g];
    }
    const int T = c->n_types;
    std::vector<double> jcost((size_t)c->n_jobs, 0.0);
    for (int j = 0; j < c->n_jobs; ++j)
        for (int g = 0; g < T; ++g) jcost[j] += icost[(size_t)j * T + g];
    std::vector<int32_t> jorder((size_t)c->n_jobs);
    std::iota(jorder.begin(), jorder.end(), 0);
    std::stable_sort(jorder.begin(), jorder.end(), [&](int a, int b) { return jcost[a] > jcost[b]; });
    std::vector<std::vector<int32_t>> qjobs(arena::kQueues);
    double qload[arena::kQueues] = {};
    for (int j : jorder) {
        int best = 0;
        for (int q = 1; q < arena::kQueues; ++q)
            if (qload[q] < qload[best]) best = q;
        qjobs[best].push_back(j);
        qload[best] += jcost[j];
    }
    std::vector<int32_t>& iorder = c->h_iorder;
    iorder.clear();
    iorder.reserve(items);
    std::vector<int32_t> types((size_t)T);
    for (int q = 0; q < arena::kQueues; ++q) {
        c->h_qoff[q] = (int32_t)iorder.size();
        for (int j : qjobs[q]) {
            std::iota(types.begin(), types.end(), 0);
            std::stable_sort(types.begin(), types.end(), [&](int a, int b) {
                return icost[(size_t)j * T + a] > icost[(size_t)j * T + b];
            });
            for (int g : types) iorder.push_back(j * T + g);
        }
    }
    c->h_qoff[arena::kQueues] = (int32_t)iorder.size();
    c->horder_valid = true;
}

arena_status upload_orders(arena_ctx* c, hipStream_t stream)
{
    compute_orders(c);
    const size_t items = (size_t)c->n_jobs * c->n_types;
    hipError_t e;
    if ((e = ensure_capacity(&c->d_item_order, &c->cap_items, items)) ||
        (e = ensure_capacity(&c->d_count_order, &c->cap_corder, (size_t)c->n_counts)))
        return fail(c, ARENA_ERR_OUT_OF_MEMORY, "work order: %s", hipGetErrorString(e));
    if ((e = hipMemcpyAsync(c->d_item_order, c->h_iorder.data(), sizeof(int32_t) * items,
                            hipMemcpyHostToDevice, stream)) ||
        (e = hipMemcpyAsync(c->d_count_order, c->h_corder.data(), sizeof(int32_t) * c->n_counts,
                            hipMemcpyHostToDevice, stream)) ||
        (e = hipStreamSynchronize(stream)))
        return hip_fail(c, e, "work order upload");
    c->order_dirty = false;
    return ARENA_OK;
}

// Library-owned device memory of one estimate, section by section, each
// section starting at a 256-byte boundary (the layout of the no-allocation
// entry point's scratch; the allocating path holds the same buffers).
struct Workspace {
    size_t counters, queue, off, batch, types, counts, kappa, items, corder, tab, pcut, total;
};

// Blocks of an estimate launch: one per resident slot (four per CU), at most
// one per item.
int estimate_blocks(const arena_ctx* c)
{
    return std::min(c->n_jobs * c->n_types, 4 * std::max(c->n_cus, 1));
}

// blocks = 0: the tables only (what the host knows before it asks the device
// for its CU count); else with the split caches of that many blocks.
Workspace workspace_layout(const arena_ctx* c, int blocks)
{
    auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
    const size_t J = (size_t)c->n_jobs, T = (size_t)c->n_types, NC = (size_t)c->n_counts;
    Workspace w;
    size_t o = 0;
    w.counters = o; o = up(o + sizeof(unsigned long long) * arena::kNumCounters);
    w.queue = o;    o = up(o + sizeof(unsigned long long) * arena::kQueues);
    w.off = o;      o = up(o + sizeof(int32_t) * (J + 1));
    w.batch = o;    o = up(o + sizeof(int32_t) * J);
    w.types = o;    o = up(o + sizeof(TypeDev) * T);
    w.counts = o;   o = up(o + sizeof(int32_t) * NC);
    w.kappa = o;    o = up(o + sizeof(float) * T * NC);
    w.items = o;    o = up(o + sizeof(int32_t) * J * T);
    w.corder = o;   o = up(o + sizeof(int32_t) * NC);
    w.tab = o;      o = up(o + (c->tab_k > 0 ? sizeof(double) * c->tab.size() : 0));
    w.pcut = o;     o = up(o + (size_t)arena::kPureCutBytes * (size_t)blocks);
    w.total = o;
    return w;
}

// Some type has one contention factor for all its counts: the kernel then
// shares every tensor-degree problem of a (job, type) across counts.
bool kappa_shared(const arena_ctx* c)
{
    if (c->n_counts < 2) return false;
    for (int g = 0; g < c->n_types; ++g) {
        bool same = true;
        for (int ci = 1; ci < c->n_counts && same; ++ci)
            same = c->kappa[(size_t)g * c->n_counts + ci] == c->kappa[(size_t)g * c->n_counts];
        if (same) return true;
    }
    return false;
}

arena_status compute_size(arena_ctx* c)
{
    if (c->size_valid) return ARENA_OK;
    // plans depend on (L, Bg) only: group jobs
    std::map<std::pair<int, int>, int64_t> groups;
    for (int j = 0; j < c->n_jobs; ++j) ++groups[{c->off[j + 1] - c->off[j], c->batch[j]}];
    arena_space_size s{};
    s.cells = (int64_t)c->n_jobs * c->n_types * c->n_counts;
    s.max_layers = c->max_layers;
    for (const auto& kv : groups) {
        for (int g = 0; g < c->n_types; ++g) {
            for (int ci = 0; ci < c->n_counts; ++ci) {
                int64_t np = plans_of_cell(c->counts[ci], c->types[g].gpn, kv.first.first,
                                           kv.first.second, c->m_values);
                s.plans += np * kv.second;
                if (np > s.max_plans_per_cell) s.max_plans_per_cell = (int32_t)np;
            }
        }
    }
    c->size = s;
    c->size_valid = true;
    return ARENA_OK;
}

}  // namespace

extern "C" {

const char* arena_status_string(arena_status s)
{
    switch (s) {
    case ARENA_OK: return "ARENA_OK";
    case ARENA_ERR_INVALID_ARG: return "ARENA_ERR_INVALID_ARG";
    case ARENA_ERR_OUT_OF_MEMORY: return "ARENA_ERR_OUT_OF_MEMORY";
    case ARENA_ERR_DEVICE: return "ARENA_ERR_DEVICE";
    case ARENA_ERR_NOT_READY: return "ARENA_ERR_NOT_READY";
    case ARENA_ERR_UNSUPPORTED: return "ARENA_ERR_UNSUPPORTED";
    }
    return "ARENA_UNKNOWN_STATUS";
}

arena_status arena_create(int hip_device, arena_ctx** out)
{
    if (!out) return ARENA_ERR_INVALID_ARG;
    *out = nullptr;
    if (hip_device < 0) return ARENA_ERR_INVALID_ARG;
    arena_ctx* c = new (std::nothrow) arena_ctx();
    if (!c) return ARENA_ERR_OUT_OF_MEMORY;
    c->device = hip_device;
    *out = c;
    return ARENA_OK;
}

void arena_destroy(arena_ctx* ctx)
{
    if (!ctx) return;
    if (ctx->dev_ready) {
        DeviceGuard g(ctx->device);
        free_device(ctx);
    }
    delete ctx;
}

const char* arena_last_error(const arena_ctx* ctx)
{
    if (!ctx) return "no context";
    return ctx->err.c_str();
}

arena_status arena_bind_jobs(arena_ctx* c, const arena_jobs_desc* d)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!d) return fail(c, ARENA_ERR_INVALID_ARG, "jobs: descriptor is NULL");
    if (d->n_jobs < 1) return fail(c, ARENA_ERR_INVALID_ARG, "jobs: n_jobs must be >= 1 (got %d)", d->n_jobs);
    if (!d->layer_offset || !d->batch)
        return fail(c, ARENA_ERR_INVALID_ARG, "jobs: layer_offset and batch (host arrays) are required");
    if (!d->t || !d->p || !d->a || !d->x || !d->a2a)
        return fail(c, ARENA_ERR_INVALID_ARG, "jobs: per-layer device arrays t, p, a, x, a2a are required");
    if (d->layer_offset[0] != 0) return fail(c, ARENA_ERR_INVALID_ARG, "jobs: layer_offset[0] must be 0");
    int maxL = 0;
    for (int j = 0; j < d->n_jobs; ++j) {
        const int L = d->layer_offset[j + 1] - d->layer_offset[j];
        if (L < 1) return fail(c, ARENA_ERR_INVALID_ARG, "jobs: job %d has %d layers", j, L);
        if (L > ARENA_MAX_LAYERS)
            return fail(c, ARENA_ERR_UNSUPPORTED, "jobs: job %d has %d layers (max %d)", j, L, ARENA_MAX_LAYERS);
        if (d->batch[j] < 1) return fail(c, ARENA_ERR_INVALID_ARG, "jobs: job %d has batch %d", j, d->batch[j]);
        if (L > maxL) maxL = L;
    }
    if (d->layer_offset[d->n_jobs] != d->n_layers_total)
        return fail(c, ARENA_ERR_INVALID_ARG, "jobs: layer_offset[n_jobs]=%d but n_layers_total=%d",
                    d->layer_offset[d->n_jobs], d->n_layers_total);
    c->n_jobs = d->n_jobs;
    c->n_layers = d->n_layers_total;
    c->max_layers = maxL;
    c->off.assign(d->layer_offset, d->layer_offset + d->n_jobs + 1);
    c->batch.assign(d->batch, d->batch + d->n_jobs);
    c->t = d->t; c->p = d->p; c->a = d->a; c->x = d->x; c->q = d->a2a;
    c->jobs_bound = true;
    c->jobs_checked = false;
    c->jobs_dirty = true;
    c->order_dirty = true;
    c->horder_valid = false;
    c->size_valid = false;
    return ARENA_OK;
}

arena_status arena_bind_grids(arena_ctx* c, const arena_grids_desc* d)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!d) return fail(c, ARENA_ERR_INVALID_ARG, "grids: descriptor is NULL");
    if (d->n_types < 1) return fail(c, ARENA_ERR_INVALID_ARG, "grids: n_types must be >= 1");
    if (d->n_types > ARENA_MAX_TYPES)
        return fail(c, ARENA_ERR_UNSUPPORTED, "grids: %d types (max %d)", d->n_types, ARENA_MAX_TYPES);
    if (d->n_counts < 1) return fail(c, ARENA_ERR_INVALID_ARG, "grids: n_counts must be >= 1");
    if (d->n_counts > ARENA_MAX_COUNTS)
        return fail(c, ARENA_ERR_UNSUPPORTED, "grids: %d counts (max %d)", d->n_counts, ARENA_MAX_COUNTS);
    if (!d->speed || !d->mem_bytes || !d->bw_intra || !d->bw_inter || !d->gpus_per_node || !d->counts)
        return fail(c, ARENA_ERR_INVALID_ARG, "grids: a host array is NULL");
    std::vector<TypeDev> ty((size_t)d->n_types);
    for (int g = 0; g < d->n_types; ++g) {
        if (!(d->speed[g] > 0.0f) || !std::isfinite(d->speed[g]))
            return fail(c, ARENA_ERR_INVALID_ARG, "grids: speed[%d] must be finite and > 0", g);
        if (!(d->mem_bytes[g] > 0.0f) || std::isnan(d->mem_bytes[g]))
            return fail(c, ARENA_ERR_INVALID_ARG, "grids: mem_bytes[%d] must be > 0", g);
        if (!is_pos_finite_or_inf(d->bw_intra[g]) || !is_pos_finite_or_inf(d->bw_inter[g]))
            return fail(c, ARENA_ERR_INVALID_ARG, "grids: bandwidths of type %d must be > 0", g);
        const int gpn = d->gpus_per_node[g];
        if (gpn < 1) return fail(c, ARENA_ERR_INVALID_ARG, "grids: gpus_per_node[%d]=%d", g, gpn);
        if (gpn > ARENA_MAX_GPUS_PER_NODE)
            return fail(c, ARENA_ERR_UNSUPPORTED, "grids: gpus_per_node[%d]=%d (max %d)", g, gpn,
                        ARENA_MAX_GPUS_PER_NODE);
        ty[g].speed = d->speed[g];
        ty[g].mem = d->mem_bytes[g];
        ty[g].bw_intra = d->bw_intra[g];
        ty[g].bw_inter = d->bw_inter[g];
        ty[g].gpn = gpn;
        ty[g].divs = 0u;
        for (int dd = 1; dd <= gpn; ++dd)
            if (gpn % dd == 0) ty[g].divs |= 1u << dd;
    }
    for (int i = 0; i < d->n_counts; ++i) {
        const int n = d->counts[i];
        if (n < 1) return fail(c, ARENA_ERR_INVALID_ARG, "grids: counts[%d]=%d", i, n);
        if (n > ARENA_MAX_GPU_COUNT)
            return fail(c, ARENA_ERR_UNSUPPORTED, "grids: counts[%d]=%d (max %d)", i, n, ARENA_MAX_GPU_COUNT);
        for (int k = 0; k < i; ++k)
            if (d->counts[k] == n) return fail(c, ARENA_ERR_INVALID_ARG, "grids: count %d listed twice", n);
    }
    c->n_types = d->n_types;
    c->n_counts = d->n_counts;
    c->types = std::move(ty);
    c->counts.assign(d->counts, d->counts + d->n_counts);
    c->kappa.assign((size_t)d->n_types * d->n_counts, 1.0f);
    c->grids_bound = true;
    c->grids_dirty = true;
    c->msets_dirty = true;
    c->kappa_dirty = true;
    c->order_dirty = true;
    c->horder_valid = false;
    c->size_valid = false;
    return ARENA_OK;
}

arena_status arena_set_kappa(arena_ctx* c, const float* kappa_host, int32_t n)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!c->grids_bound) return fail(c, ARENA_ERR_NOT_READY, "kappa: bind grids first");
    if (!kappa_host) return fail(c, ARENA_ERR_INVALID_ARG, "kappa: NULL");
    if ((int64_t)n != (int64_t)c->n_types * c->n_counts)
        return fail(c, ARENA_ERR_INVALID_ARG, "kappa: expected %d values, got %d",
                    c->n_types * c->n_counts, n);
    for (int i = 0; i < n; ++i)
        if (!(kappa_host[i] > 0.0f) || !std::isfinite(kappa_host[i]))
            return fail(c, ARENA_ERR_INVALID_ARG, "kappa[%d] must be finite and > 0", i);
    c->kappa.assign(kappa_host, kappa_host + n);
    c->kappa_dirty = true;
    return ARENA_OK;
}

arena_status arena_set_plan_space(arena_ctx* c, const int32_t* m_values, int32_t n_m, double tie_eps)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!m_values) return fail(c, ARENA_ERR_INVALID_ARG, "plan space: m_values is NULL");
    if (n_m < 1) return fail(c, ARENA_ERR_INVALID_ARG, "plan space: n_m must be >= 1");
    if (n_m > ARENA_MAX_M_VALUES)
        return fail(c, ARENA_ERR_UNSUPPORTED, "plan space: %d microbatch counts (max %d)", n_m, ARENA_MAX_M_VALUES);
    for (int i = 0; i < n_m; ++i) {
        if (m_values[i] < 1) return fail(c, ARENA_ERR_INVALID_ARG, "plan space: m_values[%d]=%d", i, m_values[i]);
        if (m_values[i] > ARENA_MAX_M)
            return fail(c, ARENA_ERR_UNSUPPORTED, "plan space: m_values[%d]=%d (max %d)", i, m_values[i], ARENA_MAX_M);
        for (int k = 0; k < i; ++k)
            if (m_values[k] == m_values[i]) return fail(c, ARENA_ERR_INVALID_ARG, "plan space: m=%d listed twice", m_values[i]);
    }
    if (!(tie_eps >= 0.0) || !(tie_eps < 1e-2))
        return fail(c, ARENA_ERR_INVALID_ARG, "plan space: tie_eps must be in [0, 1e-2)");
    c->m_values.assign(m_values, m_values + n_m);
    c->tie_eps = tie_eps;
    c->space_set = true;
    c->order_dirty = true;
    c->horder_valid = false;
    c->size_valid = false;
    return ARENA_OK;
}

arena_status arena_set_bound_pruning(arena_ctx* c, int32_t enabled)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    c->prune = enabled != 0;
    return ARENA_OK;
}

arena_status arena_set_partition_rule(arena_ctx* c, int32_t rule)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (rule != ARENA_PARTITION_BALANCED && rule != ARENA_PARTITION_MEMORY && rule != ARENA_PARTITION_EXACT_T)
        return fail(c, ARENA_ERR_INVALID_ARG, "partition rule: %d is not BALANCED (0), MEMORY (1) or EXACT_T (2)",
                    rule);
    c->partition_rule = rule;
    return ARENA_OK;
}

arena_status arena_set_comm_tables(arena_ctx* c, int32_t n_points, const double* volumes,
                                   const double* latencies)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (n_points == 0) {
        c->tab_k = 0;
        c->tab.clear();
        return ARENA_OK;
    }
    if (!c->grids_bound) return fail(c, ARENA_ERR_NOT_READY, "comm tables: bind grids first");
    if (n_points < 2 || n_points > ARENA_MAX_COMM_POINTS)
        return fail(c, ARENA_ERR_INVALID_ARG, "comm tables: %d points (2..%d)", n_points, ARENA_MAX_COMM_POINTS);
    if (!volumes || !latencies) return fail(c, ARENA_ERR_INVALID_ARG, "comm tables: NULL array");
    const size_t nt = (size_t)c->n_types * 2, K = (size_t)n_points;
    for (size_t q = 0; q < nt; ++q) {
        const double* v = volumes + q * K;
        const double* l = latencies + q * K;
        if (v[0] != 0.0)
            return fail(c, ARENA_ERR_INVALID_ARG, "comm tables: table %zu does not start at volume 0", q);
        for (size_t k = 0; k < K; ++k) {
            if (!std::isfinite(v[k]) || !std::isfinite(l[k]) || !(l[k] >= 0.0))
                return fail(c, ARENA_ERR_INVALID_ARG, "comm tables: table %zu point %zu not finite or negative", q, k);
            if (k > 0 && !(v[k] > v[k - 1]))
                return fail(c, ARENA_ERR_INVALID_ARG, "comm tables: table %zu volumes not increasing", q);
            if (k > 0 && !(l[k] >= l[k - 1]))
                return fail(c, ARENA_ERR_INVALID_ARG, "comm tables: table %zu latencies decrease", q);
        }
    }
    c->tab.assign(volumes, volumes + nt * K);
    c->tab.insert(c->tab.end(), latencies, latencies + nt * K);
    c->tab_k = n_points;
    c->tab_types = c->n_types;
    c->tab_dirty = true;
    return ARENA_OK;
}

arena_status arena_space_size_get(const arena_ctx* cc, arena_space_size* out)
{
    arena_ctx* c = const_cast<arena_ctx*>(cc);
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!out) return fail(c, ARENA_ERR_INVALID_ARG, "space size: out is NULL");
    if (!c->jobs_bound || !c->grids_bound || !c->space_set)
        return fail(c, ARENA_ERR_NOT_READY, "space size: bind jobs, grids and plan space first");
    compute_size(c);
    *out = c->size;
    return ARENA_OK;
}

arena_status arena_set_workspace_limit(arena_ctx* c, int64_t bytes)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (bytes < 0) return fail(c, ARENA_ERR_INVALID_ARG, "workspace limit: %lld bytes", (long long)bytes);
    c->ws_limit = bytes;
    return ARENA_OK;
}

}  // extern "C"

namespace {

// Host checks shared by both estimate entry points (nothing touches the device).
arena_status check_estimate(arena_ctx* c, float* t_iter, float* thr, uint32_t* plan, uint8_t* cuts,
                            int32_t cuts_stride)
{
    if (!c->jobs_bound || !c->grids_bound || !c->space_set)
        return fail(c, ARENA_ERR_NOT_READY, "estimate: bind jobs, grids and plan space first");
    if (!t_iter || !thr || !plan) return fail(c, ARENA_ERR_INVALID_ARG, "estimate: output array is NULL");
    if (cuts && cuts_stride < c->max_layers - 1)
        return fail(c, ARENA_ERR_INVALID_ARG, "estimate: cuts_stride %d < max layers - 1 = %d",
                    cuts_stride, c->max_layers - 1);
    if (cuts && cuts_stride < 1) return fail(c, ARENA_ERR_INVALID_ARG, "estimate: cuts_stride must be >= 1");
    compute_size(c);
    if (c->size.max_plans_per_cell > arena::kMaxPlans)
        return fail(c, ARENA_ERR_UNSUPPORTED, "estimate: a cell admits %d plans (max %d)",
                    c->size.max_plans_per_cell, arena::kMaxPlans);
    if (c->tab_k > 0 && c->partition_rule != ARENA_PARTITION_BALANCED)
        return fail(c, ARENA_ERR_UNSUPPORTED, "estimate: comm tables with the memory or exact-T partition rule");
    if (c->partition_rule == ARENA_PARTITION_EXACT_T && c->max_layers > arena::kExactTMaxLayers)
        return fail(c, ARENA_ERR_UNSUPPORTED, "estimate: the exact-T rule takes jobs of at most %d layers (a job has %d)",
                    arena::kExactTMaxLayers, c->max_layers);
    if (c->tab_k > 0 && c->tab_types != c->n_types)
        return fail(c, ARENA_ERR_NOT_READY, "estimate: comm tables were set for %d types, %d are bound",
                    c->tab_types, c->n_types);
    return ARENA_OK;
}

// Kernel arguments from the context, with the library-owned tables at the
// given device addresses.
arena::EstimateArgs estimate_args(const arena_ctx* c, const int32_t* d_off, const int32_t* d_batch,
                                  const TypeDev* d_types, const int32_t* d_counts, const float* d_kappa,
                                  const int32_t* d_items, const int32_t* d_corder, unsigned long long* d_queue,
                                  const double* d_tab, uint8_t* d_pcut, unsigned long long* d_counters,
                                  float* t_iter, float* thr, uint32_t* plan, uint8_t* cuts, int32_t cuts_stride)
{
    arena::EstimateArgs A;
    std::memset(&A, 0, sizeof(A));
    A.layer_offset = d_off;
    A.batch = d_batch;
    A.t = c->t; A.p = c->p; A.a = c->a; A.x = c->x; A.q = c->q;
    A.types = d_types;
    A.counts = d_counts;
    A.kappa = d_kappa;
    A.n_jobs = c->n_jobs;
    A.n_types = c->n_types;
    A.n_counts = c->n_counts;
    A.item_order = d_items;
    A.count_order = d_corder;
    A.queue = d_queue;
    for (int q = 0; q <= arena::kQueues; ++q) A.queue_off[q] = c->h_qoff[q];
    A.n_items = c->n_jobs * c->n_types;
    // one block per resident slot (four per CU); each takes items from the queue
    A.n_blocks = estimate_blocks(c);
    A.pure_cuts = d_pcut;
    A.share_tp = kappa_shared(c) ? 1 : 0;
    // ascending: the kernel bisects the microbatch counts for the memory limit
    std::vector<int32_t> ms(c->m_values);
    std::sort(ms.begin(), ms.end());
    A.n_m = (int32_t)ms.size();
    for (int i = 0; i < A.n_m; ++i) A.m_values[i] = ms[i];
    A.tie_eps = c->tie_eps;
    A.prune = c->prune ? 1 : 0;
    A.mem_rule = c->partition_rule == ARENA_PARTITION_MEMORY ? 1 : 0;
    A.exact_t = c->partition_rule == ARENA_PARTITION_EXACT_T ? 1 : 0;
    if (c->tab_k > 0) {
        A.tab_k = c->tab_k;
        A.tab_vol = d_tab;
        A.tab_lat = d_tab + c->tab.size() / 2;
    }
    A.t_iter = t_iter;
    A.thr = thr;
    A.plan = plan;
    A.cuts = cuts;
    A.cuts_stride = cuts ? cuts_stride : 0;
    A.counters = d_counters;
    return A;
}

}  // namespace

extern "C" {

arena_status arena_estimate(arena_ctx* c, float* t_iter, float* thr, uint32_t* plan, uint8_t* cuts,
                            int32_t cuts_stride, void* stream_ptr)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    arena_status st = check_estimate(c, t_iter, thr, plan, cuts, cuts_stride);
    if (st != ARENA_OK) return st;
    // the tables (known on the host), then with the blocks' split caches (their
    // number needs the device's CU count)
    const Workspace ws0 = workspace_layout(c, 0);
    if (c->ws_limit > 0 && ws0.total > (size_t)c->ws_limit)
        return fail(c, ARENA_ERR_OUT_OF_MEMORY,
                    "estimate: its tables alone need %zu bytes of device workspace (limit %lld)", ws0.total,
                    (long long)c->ws_limit);
    hipStream_t stream = (hipStream_t)stream_ptr;
    DeviceGuard guard(c->device);
    if (guard.status != hipSuccess) return hip_fail(c, guard.status, "hipSetDevice");
    hipError_t e;
    if (c->n_cus == 0 &&
        (e = hipDeviceGetAttribute(&c->n_cus, hipDeviceAttributeMultiprocessorCount, c->device)))
        return hip_fail(c, e, "hipDeviceGetAttribute");
    const Workspace ws = workspace_layout(c, estimate_blocks(c));
    if (c->ws_limit > 0 && ws.total > (size_t)c->ws_limit)
        return fail(c, ARENA_ERR_OUT_OF_MEMORY, "estimate: needs %zu bytes of device workspace (limit %lld)",
                    ws.total, (long long)c->ws_limit);
    st = ensure_device(c, stream);
    if (st != ARENA_OK) return st;
    if ((e = ensure_capacity(&c->d_pcut, &c->cap_pcut, (size_t)arena::kPureCutBytes * estimate_blocks(c))))
        return fail(c, ARENA_ERR_OUT_OF_MEMORY, "split caches: %s", hipGetErrorString(e));
    if (c->order_dirty && (st = upload_orders(c, stream)) != ARENA_OK) return st;
    if (c->tab_k > 0) {
        if (c->tab_dirty) {
            if ((e = ensure_capacity(&c->d_tab, &c->cap_tab, c->tab.size())))
                return fail(c, ARENA_ERR_OUT_OF_MEMORY, "comm tables: %s", hipGetErrorString(e));
            if ((e = hipMemcpyAsync(c->d_tab, c->tab.data(), sizeof(double) * c->tab.size(),
                                    hipMemcpyHostToDevice, stream)) ||
                (e = hipStreamSynchronize(stream)))
                return hip_fail(c, e, "comm table upload");
            c->tab_dirty = false;
        }
    }
    const arena::EstimateArgs A =
        estimate_args(c, c->d_off, c->d_batch, c->d_types, c->d_counts, c->d_kappa, c->d_item_order,
                      c->d_count_order, c->d_queue, c->d_tab, c->d_pcut, c->d_counters, t_iter, thr, plan, cuts,
                      cuts_stride);
    if ((e = arena::launch_zero_counters(c->d_counters, arena::kNumCounters, stream)) ||
        (e = arena::launch_zero_counters(c->d_queue, arena::kQueues, stream)))
        return hip_fail(c, e, "counter reset");
    if ((e = arena::launch_estimate(A, stream))) return hip_fail(c, e, "estimate launch");
    c->last_counters = c->d_counters;
    c->last_space_plans = c->size.plans;
    return ARENA_OK;
}

arena_status arena_estimate_noalloc(arena_ctx* c, float* t_iter, float* thr, uint32_t* plan, uint8_t* cuts,
                                    int32_t cuts_stride, void* stream_ptr)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    arena_status st = check_estimate(c, t_iter, thr, plan, cuts, cuts_stride);
    if (st != ARENA_OK) return st;
    // the tables (known on the host), then with the blocks' split caches (their
    // number needs the device's CU count)
    const Workspace ws0 = workspace_layout(c, 0);
    if (ws0.total > arena::kNoallocScratchBytes)
        return fail(c, ARENA_ERR_OUT_OF_MEMORY,
                    "estimate_noalloc: the bound workload's tables alone need %zu bytes of scratch (max %zu): "
                    "use arena_estimate", ws0.total, (size_t)arena::kNoallocScratchBytes);
    hipStream_t stream = (hipStream_t)stream_ptr;
    DeviceGuard guard(c->device);
    if (guard.status != hipSuccess) return hip_fail(c, guard.status, "hipSetDevice");
    hipError_t e;
    if (c->n_cus == 0 &&
        (e = hipDeviceGetAttribute(&c->n_cus, hipDeviceAttributeMultiprocessorCount, c->device)))
        return hip_fail(c, e, "hipDeviceGetAttribute");
    const Workspace ws = workspace_layout(c, estimate_blocks(c));
    if (ws.total > arena::kNoallocScratchBytes)
        return fail(c, ARENA_ERR_OUT_OF_MEMORY,
                    "estimate_noalloc: the bound workload needs %zu bytes of scratch (max %zu): "
                    "use arena_estimate", ws.total, (size_t)arena::kNoallocScratchBytes);
    char* base = nullptr;
    if ((e = arena::scratch_address(c->device, (void**)&base))) return hip_fail(c, e, "scratch address");
    auto* d_counters = (unsigned long long*)(base + ws.counters);
    auto* d_queue = (unsigned long long*)(base + ws.queue);
    auto* d_off = (int32_t*)(base + ws.off);
    auto* d_batch = (int32_t*)(base + ws.batch);
    auto* d_types = (TypeDev*)(base + ws.types);
    auto* d_counts = (int32_t*)(base + ws.counts);
    auto* d_kappa = (float*)(base + ws.kappa);
    auto* d_items = (int32_t*)(base + ws.items);
    auto* d_corder = (int32_t*)(base + ws.corder);
    auto* d_tab = (double*)(base + ws.tab);
    auto* d_pcut = (uint8_t*)(base + ws.pcut);
    compute_orders(c);
    const size_t J = (size_t)c->n_jobs, T = (size_t)c->n_types, NC = (size_t)c->n_counts;
    // the scratch is shared by every call on this device: every table is
    // copied again (pageable host sources: each copy has read its source
    // when it returns)
    if ((e = hipMemcpyAsync(d_off, c->off.data(), sizeof(int32_t) * (J + 1), hipMemcpyHostToDevice, stream)) ||
        (e = hipMemcpyAsync(d_batch, c->batch.data(), sizeof(int32_t) * J, hipMemcpyHostToDevice, stream)))
        return hip_fail(c, e, "job table copy");
    if (!c->jobs_checked) {
        arena::ValidateArgs v;
        v.layer_offset = d_off;
        v.n_jobs = c->n_jobs;
        v.arrays[0] = c->t; v.arrays[1] = c->p; v.arrays[2] = c->a; v.arrays[3] = c->x; v.arrays[4] = c->q;
        v.bad = d_counters;
        unsigned long long bad = 0;
        if ((e = arena::launch_zero_counters(d_counters, 1, stream)) || (e = arena::launch_validate(v, stream)) ||
            (e = hipMemcpyAsync(&bad, d_counters, sizeof(bad), hipMemcpyDeviceToHost, stream)) ||
            (e = hipStreamSynchronize(stream)))
            return hip_fail(c, e, "job value check");
        if (bad != 0)
            return fail(c, ARENA_ERR_INVALID_ARG, "jobs: %llu per-layer values are negative or not finite", bad);
        c->jobs_checked = true;
    }
    if ((e = hipMemcpyAsync(d_types, c->types.data(), sizeof(TypeDev) * T, hipMemcpyHostToDevice, stream)) ||
        (e = hipMemcpyAsync(d_counts, c->counts.data(), sizeof(int32_t) * NC, hipMemcpyHostToDevice, stream)) ||
        (e = hipMemcpyAsync(d_kappa, c->kappa.data(), sizeof(float) * T * NC, hipMemcpyHostToDevice, stream)) ||
        (e = hipMemcpyAsync(d_items, c->h_iorder.data(), sizeof(int32_t) * J * T, hipMemcpyHostToDevice,
                            stream)) ||
        (e = hipMemcpyAsync(d_corder, c->h_corder.data(), sizeof(int32_t) * NC, hipMemcpyHostToDevice, stream)))
        return hip_fail(c, e, "table copy");
    if (c->tab_k > 0 &&
        (e = hipMemcpyAsync(d_tab, c->tab.data(), sizeof(double) * c->tab.size(), hipMemcpyHostToDevice, stream)))
        return hip_fail(c, e, "comm table copy");
    const arena::EstimateArgs A = estimate_args(c, d_off, d_batch, d_types, d_counts, d_kappa, d_items, d_corder,
                                                d_queue, d_tab, d_pcut, d_counters, t_iter, thr, plan, cuts,
                                                cuts_stride);
    // zeroed by a kernel, not a memset node
    if ((e = arena::launch_zero_counters(d_counters, arena::kNumCounters, stream)) ||
        (e = arena::launch_zero_counters(d_queue, arena::kQueues, stream)))
        return hip_fail(c, e, "counter reset");
    if ((e = arena::launch_estimate(A, stream))) return hip_fail(c, e, "estimate launch");
    c->last_counters = d_counters;
    c->last_space_plans = c->size.plans;
    return ARENA_OK;
}

arena_status arena_get_counters(arena_ctx* c, arena_counters* out)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!out) return fail(c, ARENA_ERR_INVALID_ARG, "counters: out is NULL");
    if (!c->last_counters) return fail(c, ARENA_ERR_NOT_READY, "counters: no estimate has run");
    DeviceGuard guard(c->device);
    if (guard.status != hipSuccess) return hip_fail(c, guard.status, "hipSetDevice");
    hipError_t e;
    if ((e = hipDeviceSynchronize())) return hip_fail(c, e, "synchronise");
    unsigned long long h[arena::kNumCounters];
    if ((e = hipMemcpy(h, c->last_counters, sizeof(h), hipMemcpyDeviceToHost)))
        return hip_fail(c, e, "counter copy");
    out->cells = (int64_t)h[arena::kCells];
    out->plans = (int64_t)h[arena::kPlans];
    out->problems = (int64_t)h[arena::kProblems];
    out->dp_entries = (int64_t)h[arena::kDpEntries];
    out->infeasible_cells = (int64_t)h[arena::kInfeasible];
    // every plan of the space is priced or skipped (the kernels count the priced)
    out->plans_skipped = c->last_space_plans - out->plans;
    out->alg_ops = (int64_t)h[arena::kAlgOps];
    out->mem_partitions = (int64_t)h[arena::kMemParts];
    if (h[arena::kOverflow]) return fail(c, ARENA_ERR_UNSUPPORTED, "counters: plan buffer overflow");
    return ARENA_OK;
}

}  // extern "C"

namespace {

// Multisets of s powers of two summing to n (exponents non-increasing,
// packed 4 bits per position, largest first), in lexicographically
// descending order.
void pow2_multisets(int n, int s, int k, int maxe, unsigned long long cur, std::vector<unsigned long long>& out)
{
    if (k == s) {
        if (n == 0) out.push_back(cur);
        return;
    }
    const int left = s - k - 1;
    for (int e = maxe; e >= 0; --e) {
        const int v = 1 << e;
        if (v > n - left) continue;
        if ((long long)(left + 1) * v < n) break;     // the rest take at most v each
        pow2_multisets(n - v, s, k + 1, e, cur | ((unsigned long long)e << (4 * k)), out);
    }
}

arena_status build_msets(arena_ctx* c)
{
    c->msets.clear();
    c->mset_off.assign((size_t)c->n_counts * 17 + 1, 0);
    for (int ci = 0; ci < c->n_counts; ++ci) {
        const int n = c->counts[ci];
        int maxe = 0;
        while ((1 << (maxe + 1)) <= n) ++maxe;
        for (int s = 0; s < 17; ++s) {
            c->mset_off[(size_t)ci * 17 + s] = (int32_t)c->msets.size();
            if (s == 0) continue;
            const size_t before = c->msets.size();
            pow2_multisets(n, s, 0, maxe, 0ull, c->msets);
            if (c->msets.size() - before > (size_t)arena::kProxyMaxMultisets)
                return fail(c, ARENA_ERR_UNSUPPORTED, "proxy: %zu power-of-two splits of %d GPUs into %d stages (max %d)",
                            c->msets.size() - before, n, s, arena::kProxyMaxMultisets);
        }
    }
    c->mset_off[(size_t)c->n_counts * 17] = (int32_t)c->msets.size();
    return ARENA_OK;
}

}  // namespace

extern "C" {

arena_status arena_proxy_estimate(arena_ctx* c, const arena_proxy_desc* d, float* t_iter, float* thr,
                                  uint64_t* plan, void* stream_ptr)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!c->jobs_bound || !c->grids_bound || !c->space_set)
        return fail(c, ARENA_ERR_NOT_READY, "proxy: bind jobs, grids and plan space first");
    if (!d) return fail(c, ARENA_ERR_INVALID_ARG, "proxy: descriptor is NULL");
    if (!t_iter || !thr || !plan) return fail(c, ARENA_ERR_INVALID_ARG, "proxy: output array is NULL");
    if (!d->hbm_bw) return fail(c, ARENA_ERR_INVALID_ARG, "proxy: hbm_bw is NULL");
    if (!(d->f_ref > 0.0) || !std::isfinite(d->f_ref))
        return fail(c, ARENA_ERR_INVALID_ARG, "proxy: f_ref must be finite and > 0");
    if (d->n_ops < 1 || d->n_ops > ARENA_MAX_PROXY_OPS)
        return fail(c, ARENA_ERR_INVALID_ARG, "proxy: n_ops=%d not in 1..%d", d->n_ops, ARENA_MAX_PROXY_OPS);
    if ((long long)c->n_jobs * c->n_types * c->n_counts > 0x7fffffffLL)
        return fail(c, ARENA_ERR_UNSUPPORTED, "proxy: more than 2^31-1 cells");
    std::vector<double> hbm((size_t)c->n_types);
    for (int g = 0; g < c->n_types; ++g) {
        if (!(d->hbm_bw[g] > 0.0f) || !std::isfinite(d->hbm_bw[g]))
            return fail(c, ARENA_ERR_INVALID_ARG, "proxy: hbm_bw[%d] must be finite and > 0", g);
        hbm[g] = (double)d->hbm_bw[g];
    }
    arena_status st;
    if (c->msets_dirty && (st = build_msets(c)) != ARENA_OK) return st;
    hipStream_t stream = (hipStream_t)stream_ptr;
    DeviceGuard guard(c->device);
    if (guard.status != hipSuccess) return hip_fail(c, guard.status, "hipSetDevice");
    if ((st = ensure_device(c, stream)) != ARENA_OK) return st;
    hipError_t e;
    if (c->msets_dirty) {
        if ((e = ensure_capacity(&c->d_msets, &c->cap_msets, c->msets.size())) ||
            (e = ensure_capacity(&c->d_mset_off, &c->cap_mset_off, c->mset_off.size())))
            return fail(c, ARENA_ERR_OUT_OF_MEMORY, "proxy tables: %s", hipGetErrorString(e));
        if ((e = hipMemcpyAsync(c->d_msets, c->msets.data(), sizeof(unsigned long long) * c->msets.size(),
                                hipMemcpyHostToDevice, stream)) ||
            (e = hipMemcpyAsync(c->d_mset_off, c->mset_off.data(), sizeof(int32_t) * c->mset_off.size(),
                                hipMemcpyHostToDevice, stream)) ||
            (e = hipStreamSynchronize(stream)))
            return hip_fail(c, e, "proxy table upload");
        c->msets_dirty = false;
    }
    if ((e = ensure_capacity(&c->d_hbm, &c->cap_hbm, hbm.size())))
        return fail(c, ARENA_ERR_OUT_OF_MEMORY, "proxy bandwidths: %s", hipGetErrorString(e));
    if ((e = hipMemcpyAsync(c->d_hbm, hbm.data(), sizeof(double) * hbm.size(), hipMemcpyHostToDevice, stream)) ||
        (e = hipStreamSynchronize(stream)))
        return hip_fail(c, e, "proxy bandwidth upload");

    arena::ProxyArgs A;
    std::memset(&A, 0, sizeof(A));
    A.layer_offset = c->d_off;
    A.batch = c->d_batch;
    A.t = c->t; A.p = c->p; A.a = c->a; A.x = c->x; A.q = c->q;
    A.types = c->d_types;
    A.hbm = c->d_hbm;
    A.counts = c->d_counts;
    A.kappa = c->d_kappa;
    A.msets = c->d_msets;
    A.mset_off = c->d_mset_off;
    A.n_jobs = c->n_jobs;
    A.n_types = c->n_types;
    A.n_counts = c->n_counts;
    A.n_ops = d->n_ops;
    A.n_m = (int32_t)c->m_values.size();
    for (int i = 0; i < A.n_m; ++i) A.m_values[i] = c->m_values[i];
    A.tie_eps = c->tie_eps;
    A.f_ref = d->f_ref;
    A.t_iter = t_iter;
    A.thr = thr;
    A.plan = (unsigned long long*)plan;
    A.queue = c->d_queue;
    A.n_cus = c->n_cus;
    if ((e = arena::launch_zero_counters(c->d_queue, 1, stream)))
        return hip_fail(c, e, "proxy queue reset");
    if ((e = arena::launch_proxy(A, stream))) return hip_fail(c, e, "proxy launch");
    return ARENA_OK;
}

arena_status arena_schedule(arena_ctx* c, const arena_sched_desc* d, void* stream_ptr)
{
    if (!c) return ARENA_ERR_INVALID_ARG;
    c->err.clear();
    if (!d) return fail(c, ARENA_ERR_INVALID_ARG, "schedule: descriptor is NULL");
    if (d->n_jobs < 0) return fail(c, ARENA_ERR_INVALID_ARG, "schedule: n_jobs=%d", d->n_jobs);
    if (d->n_jobs > ARENA_MAX_SCHED_JOBS)
        return fail(c, ARENA_ERR_UNSUPPORTED, "schedule: %d jobs (max %d)", d->n_jobs, ARENA_MAX_SCHED_JOBS);
    if (d->n_types < 1) return fail(c, ARENA_ERR_INVALID_ARG, "schedule: n_types must be >= 1");
    if (d->n_types > ARENA_MAX_TYPES)
        return fail(c, ARENA_ERR_UNSUPPORTED, "schedule: %d types (max %d)", d->n_types, ARENA_MAX_TYPES);
    if (d->n_counts < 1) return fail(c, ARENA_ERR_INVALID_ARG, "schedule: n_counts must be >= 1");
    if (d->n_counts > ARENA_MAX_COUNTS)
        return fail(c, ARENA_ERR_UNSUPPORTED, "schedule: %d counts (max %d)", d->n_counts, ARENA_MAX_COUNTS);
    if (d->n_queue < 0 || d->n_queue > d->n_jobs)
        return fail(c, ARENA_ERR_INVALID_ARG, "schedule: n_queue=%d not in 0..n_jobs", d->n_queue);
    if (d->depth < 1 || d->depth > ARENA_MAX_SCHED_DEPTH)
        return fail(c, ARENA_ERR_INVALID_ARG, "schedule: depth=%d not in 1..%d", d->depth, ARENA_MAX_SCHED_DEPTH);
    if (!d->counts || !d->capacity) return fail(c, ARENA_ERR_INVALID_ARG, "schedule: a host array is NULL");
    if (!d->result || (d->n_jobs > 0 && (!d->thr || !d->alloc_type || !d->alloc_count)) ||
        (d->n_queue > 0 && (!d->queue || !d->priority || !d->launched)))
        return fail(c, ARENA_ERR_INVALID_ARG, "schedule: a device array is NULL");
    if (d->objective != ARENA_SCHED_THROUGHPUT && d->objective != ARENA_SCHED_FAIRNESS)
        return fail(c, ARENA_ERR_INVALID_ARG, "schedule: objective=%d is neither throughput (0) nor fairness (1)",
                    d->objective);
    const int n_ddl = (d->batch != nullptr) + (d->iters != nullptr) + (d->deadline != nullptr);
    if (d->objective == ARENA_SCHED_FAIRNESS) {
        if (!d->batch || !d->iters)
            return fail(c, ARENA_ERR_INVALID_ARG, "schedule: the fairness objective needs batch and iters");
    } else if (n_ddl != 0 && n_ddl != 3) {
        return fail(c, ARENA_ERR_INVALID_ARG, "schedule: give batch, iters and deadline together or none");
    }
    for (int i = 0; i < d->n_counts; ++i) {
        const int n = d->counts[i];
        if (n < 1 || n > ARENA_MAX_GPU_COUNT)
            return fail(c, ARENA_ERR_INVALID_ARG, "schedule: counts[%d]=%d not in 1..%d", i, n, ARENA_MAX_GPU_COUNT);
        if (i > 0 && n <= d->counts[i - 1])
            return fail(c, ARENA_ERR_INVALID_ARG, "schedule: counts must be strictly ascending");
    }
    for (int g = 0; g < d->n_types; ++g)
        if (d->capacity[g] < 0 || d->capacity[g] > ARENA_MAX_SCHED_CAPACITY)
            return fail(c, ARENA_ERR_INVALID_ARG, "schedule: capacity[%d]=%d not in 0..%d", g, d->capacity[g],
                        ARENA_MAX_SCHED_CAPACITY);
    hipStream_t stream = (hipStream_t)stream_ptr;
    DeviceGuard guard(c->device);
    if (guard.status != hipSuccess) return hip_fail(c, guard.status, "hipSetDevice");
    hipError_t e;
    const size_t n = (size_t)arena::kMaxSchedCounts + arena::kMaxSchedTypes;
    if (!c->sched_done && (e = hipEventCreateWithFlags(&c->sched_done, hipEventDisableTiming)))
        return hip_fail(c, e, "hipEventCreate");
    if ((e = ensure_capacity(&c->d_sched, &c->cap_sched, n)))
        return fail(c, ARENA_ERR_OUT_OF_MEMORY, "schedule tables: %s", hipGetErrorString(e));
    if (!c->h_sched) {
        if ((e = hipHostMalloc((void**)&c->h_sched, sizeof(int32_t) * n, 0)))
            return fail(c, ARENA_ERR_OUT_OF_MEMORY, "pinned schedule staging");
        c->cap_hsched = n;
    }
    // the previous call's upload must have left the staging buffer
    if ((e = hipEventSynchronize(c->sched_done))) return hip_fail(c, e, "schedule staging wait");
    std::memcpy(c->h_sched, d->counts, sizeof(int32_t) * d->n_counts);
    std::memcpy(c->h_sched + arena::kMaxSchedCounts, d->capacity, sizeof(int32_t) * d->n_types);
    if ((e = hipMemcpyAsync(c->d_sched, c->h_sched, sizeof(int32_t) * n, hipMemcpyHostToDevice, stream)) ||
        (e = hipEventRecord(c->sched_done, stream)))
        return hip_fail(c, e, "schedule table upload");
    arena::SchedArgs A;
    std::memset(&A, 0, sizeof(A));
    A.thr = d->thr;
    A.counts = c->d_sched;
    A.capacity = c->d_sched + arena::kMaxSchedCounts;
    A.alloc_type = d->alloc_type;
    A.alloc_count = d->alloc_count;
    A.queue = d->queue;
    A.priority = d->priority;
    A.launched = d->launched;
    A.result = d->result;
    A.n_jobs = d->n_jobs;
    A.n_types = d->n_types;
    A.n_counts = d->n_counts;
    A.n_queue = d->n_queue;
    A.depth = d->depth;
    if (d->n_jobs > 0 && (n_ddl == 3 || d->objective == ARENA_SCHED_FAIRNESS)) {
        A.batch = d->batch;
        A.iters = d->iters;
        A.ddl = d->deadline;        // NULL: no deadline constraint
    }
    A.objective = d->objective;
    if ((e = arena::launch_schedule(A, stream))) return hip_fail(c, e, "schedule launch");
    return ARENA_OK;
}

}  // extern "C"
