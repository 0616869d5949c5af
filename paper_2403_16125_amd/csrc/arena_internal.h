// Internal interface between the host side of the C ABI and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace arena {

constexpr int kWave = 64;
constexpr int kLmax = 128;          // layers per job
constexpr int kMaxTargets = 32;     // pipeline degrees per partition problem (<= 26 for n <= 1024)
constexpr int kMaxPlans = 256;      // plans per cell
constexpr int kMaxM = 16;           // microbatch choices
constexpr int kWavesPerBlock = 4;   // waves of one (job, type) block, each on its own cells
constexpr int kMaxDp = 1024;        // largest data-parallel degree (counts are <= 1024)
constexpr int kMaxTabPoints = 16;   // samples per communication latency table
constexpr int kExactTMaxLayers = 96; // layers per job under the exact-T rule
constexpr int kQueues = 8;          // item queues, one per XCD (each XCD has its own L2)

// GPU type as the kernels read it (doubles converted from the f32 inputs).
struct TypeDev {
    double speed, mem, bw_intra, bw_inter;
    int32_t gpn;
    uint32_t divs;    // bit d: d divides gpn (gpn <= 31)
};

// Device tallies, zeroed before each estimate.
enum Counter { kCells = 0, kPlans, kProblems, kDpEntries, kInfeasible, kOverflow, kAlgOps, kMemParts,
               kNumCounters };

// Bytes of one block's cache of the pure-compute problem's canonical splits:
// row pp (2 <= pp <= 128) holds the cuts c_0 .. c_pp, one byte each, from
// byte pp (pp + 1) / 2 - 3.
constexpr int kPureCutBytes = 8448;

struct EstimateArgs {
    const int32_t* layer_offset;  // [J+1]
    const int32_t* batch;         // [J]
    const float* t;
    const float* p;
    const float* a;
    const float* x;
    const float* q;               // all-to-all bytes per sample
    const TypeDev* types;         // [T]
    const int32_t* counts;        // [NC]
    const float* kappa;           // [T*NC]
    const int32_t* item_order;    // [J*T] (job, type) items: queue q holds [queue_off[q], queue_off[q+1])
    unsigned long long* queue;    // [kQueues] next item of each queue (zeroed before each launch)
    int32_t queue_off[kQueues + 1];
    int32_t n_items;              // J * T
    int32_t n_blocks;             // resident blocks launched; each takes items until none is left
    uint8_t* pure_cuts;           // [n_blocks * kPureCutBytes] each block's cache of pure-compute splits
    const int32_t* count_order;   // [NC] count indices, largest count first
    int32_t n_jobs, n_types, n_counts;
    int32_t share_tp;             // some type has one kappa for all its counts: share tp problems
    int32_t n_m;
    int32_t m_values[kMaxM];
    double tie_eps;
    int32_t prune;                // bound pruning on
    int32_t mem_rule;             // partition rule 1: balanced among the splits that fit memory
    int32_t exact_t;              // partition rule 2: the split of least iteration time that fits memory
    // interpolated communication latency: tab_k points per (type, link),
    // volumes then latencies, each [T][2][tab_k]; tab_k = 0: volume / bandwidth
    const double* tab_vol;
    const double* tab_lat;
    int32_t tab_k;
    float* t_iter;
    float* thr;
    uint32_t* plan;
    uint8_t* cuts;                // nullable
    int32_t cuts_stride;
    unsigned long long* counters; // [kNumCounters]
};

struct ValidateArgs {
    const int32_t* layer_offset;
    int32_t n_jobs;
    const float* arrays[5];
    unsigned long long* bad;      // [1] count of non-finite or negative values
};

// Proxy-plan planner (arena_proxy_estimate).
constexpr int kProxyMaxOps = 16;            // clustered operators per job
constexpr int kProxyMaxMultisets = 1280;    // power-of-two multisets of one (count, stage count)
constexpr int kProxyPlanWords = 3;          // u64 words of plan per cell

struct ProxyArgs {
    const int32_t* layer_offset;  // [J+1]
    const int32_t* batch;         // [J]
    const float* t;
    const float* p;
    const float* a;
    const float* x;
    const float* q;               // all-to-all bytes per sample
    const TypeDev* types;         // [T]
    const double* hbm;            // [T] memory bandwidth, bytes/s
    const int32_t* counts;        // [NC]
    const float* kappa;           // [T*NC]
    // multisets of s powers of two summing to counts[c], exponents at bits
    // 4k (k-th largest), lexicographically descending; (c, s) spans
    // msets[mset_off[c*17 + s] .. mset_off[c*17 + s + 1])
    const unsigned long long* msets;
    const int32_t* mset_off;      // [NC*17 + 1]
    int32_t n_jobs, n_types, n_counts, n_ops;
    int32_t n_m;
    int32_t m_values[kMaxM];
    double tie_eps, f_ref;
    float* t_iter;
    float* thr;
    unsigned long long* plan;     // [C * kProxyPlanWords]
    unsigned long long* queue;    // [1] next cell to take (zeroed before each launch)
    int32_t n_cus;                // compute units: one launch fills them with resident blocks
};

hipError_t launch_proxy(const ProxyArgs& args, hipStream_t stream);

// One scheduling step over the throughput matrix (arena_schedule).
constexpr int kMaxSchedTypes = 64;
constexpr int kMaxSchedCounts = 512;
constexpr int kMaxSchedDepth = 256;
constexpr int kMaxSchedJobs = 65536;

struct SchedArgs {
    const float* thr;             // [J * T * NC]
    const int32_t* counts;        // [NC] device copy, strictly ascending
    const int32_t* capacity;      // [T] device copy
    int32_t* alloc_type;          // [J] in/out
    int32_t* alloc_count;         // [J] in/out
    const int32_t* queue;         // [Q]
    const int32_t* priority;      // [Q]
    int32_t* launched;            // [Q] out
    int32_t* result;              // [8] out: status, moves, decisions, candidates examined
    int32_t n_jobs, n_types, n_counts, n_queue, depth;
    // deadline constraint (Eq. 6): all null, or per job batch, remaining
    // iterations and time left to the deadline
    const int32_t* batch;
    const float* iters;
    const float* ddl;
    int32_t objective;            // 0 throughput (Eq. 5), 1 finish-time fairness (Eq. 7)
};

hipError_t launch_estimate(const EstimateArgs& args, hipStream_t stream);

// Scratch of the no-allocation estimate: a statically sized device array,
// one copy per device.  scratch_address returns its device address on
// `device`, which must be the current device (looked up once per device).
constexpr size_t kNoallocScratchBytes = size_t(16) << 20;
constexpr int kMaxScratchDevices = 64;
hipError_t scratch_address(int device, void** out);
hipError_t launch_schedule(const SchedArgs& args, hipStream_t stream);
hipError_t launch_zero_counters(unsigned long long* counters, int n, hipStream_t stream);
hipError_t launch_validate(const ValidateArgs& args, hipStream_t stream);

}  // namespace arena
