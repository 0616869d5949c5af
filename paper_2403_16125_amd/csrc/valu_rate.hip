// Issue-rate microbenchmark of the VALU operations the estimate kernels are
// built from, in double and in float.  The estimate kernels keep every cost,
// prefix and recursion value in fp64; this measures, on the GPU they run on,
// what each operation class costs in fp64 against fp32 when compiled the way
// the library is (no packed fp32 instructions).
//
// Each thread runs eight independent dependency chains (enough to hide the
// VALU latency at eight waves per SIMD), so the kernel is bound by issue
// rate.  Operation classes:
//   0 fma     x = fma(x, a, b)
//   1 add     x = x + b
//   2 minmax  x = max(min(x, a), b)                       (two operations)
//   3 select  x = (x >= a - y) ? x - b : y                 (the recursion's
//             crossing test: subtract, compare, select; y = x + b)
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

constexpr int kChains = 8;
constexpr int kThreads = 256;

__device__ __forceinline__ float fma_t(float a, float b, float c) { return fmaf(a, b, c); }
__device__ __forceinline__ double fma_t(double a, double b, double c) { return fma(a, b, c); }
__device__ __forceinline__ float min_t(float a, float b) { return fminf(a, b); }
__device__ __forceinline__ double min_t(double a, double b) { return fmin(a, b); }
__device__ __forceinline__ float max_t(float a, float b) { return fmaxf(a, b); }
__device__ __forceinline__ double max_t(double a, double b) { return fmax(a, b); }

template <typename T, int OP>
__global__ __launch_bounds__(kThreads) void rate_kernel(T* out, int iters, T a, T b)
{
    const int gid = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    T x[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) x[k] = (T)(gid % 977 + k) * (T)0.001;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < kChains; ++k) {
            if (OP == 0) {
                x[k] = fma_t(x[k], a, b);
            } else if (OP == 1) {
                x[k] = x[k] + b;
            } else if (OP == 2) {
                x[k] = max_t(min_t(x[k], a), b);
            } else {
                const T y = x[k] + b;
                x[k] = (x[k] >= a - y) ? x[k] - b : y;
            }
        }
    }
    T s = (T)0;
#pragma unroll
    for (int k = 0; k < kChains; ++k) s = s + x[k];
    out[gid] = s;
}

template <typename T>
hipError_t launch(int op, int blocks, int iters, void* out, hipStream_t st)
{
    const T a = (T)0.75, b = (T)0.125;
    T* o = (T*)out;
    switch (op) {
    case 0: hipLaunchKernelGGL((rate_kernel<T, 0>), dim3(blocks), dim3(kThreads), 0, st, o, iters, a, b); break;
    case 1: hipLaunchKernelGGL((rate_kernel<T, 1>), dim3(blocks), dim3(kThreads), 0, st, o, iters, a, b); break;
    case 2: hipLaunchKernelGGL((rate_kernel<T, 2>), dim3(blocks), dim3(kThreads), 0, st, o, iters, a, b); break;
    default: hipLaunchKernelGGL((rate_kernel<T, 3>), dim3(blocks), dim3(kThreads), 0, st, o, iters, a, b); break;
    }
    return hipGetLastError();
}

}  // namespace

// Runs operation class `op` (0..3) in double (is_double != 0) or float over
// `blocks` blocks of 256 threads, `iters` steps per chain: one untimed launch,
// then `reps` timed launches; ms_out[r] receives each launch's time.  Returns
// 0 or the HIP error code.  Allocates and frees its own output buffer.
extern "C" int valu_rate_run(int op, int is_double, int blocks, int iters, int reps, double* ms_out)
{
    if (op < 0 || op > 3 || blocks <= 0 || iters <= 0 || reps <= 0 || !ms_out) return (int)hipErrorInvalidValue;
    void* out = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    const size_t bytes = (size_t)blocks * kThreads * (is_double ? sizeof(double) : sizeof(float));
    hipError_t e = hipMalloc(&out, bytes);
    if (e == hipSuccess) e = hipEventCreate(&e0);
    if (e == hipSuccess) e = hipEventCreate(&e1);
    for (int r = -1; e == hipSuccess && r < reps; ++r) {
        if ((e = hipEventRecord(e0, nullptr)) != hipSuccess) break;
        e = is_double ? launch<double>(op, blocks, iters, out, nullptr) : launch<float>(op, blocks, iters, out, nullptr);
        if (e != hipSuccess) break;
        if ((e = hipEventRecord(e1, nullptr)) != hipSuccess || (e = hipEventSynchronize(e1)) != hipSuccess) break;
        float ms = 0.0f;
        if ((e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess) break;
        if (r >= 0) ms_out[r] = (double)ms;
    }
    if (e1) (void)hipEventDestroy(e1);
    if (e0) (void)hipEventDestroy(e0);
    if (out) (void)hipFree(out);
    return (int)e;
}
