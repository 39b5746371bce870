// Measured ceilings of the GPU: the int32 VALU rate and the copy bandwidth (rk_calib.h).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rk_calib.h"

namespace {

constexpr int CHAINS = 8;

// Eight independent add-then-min chains per lane.  The empty asm keeps each step's value
// live in a register, so the compiler cannot fold steps together or solve the chain.
__global__ __launch_bounds__(256) void k_valu(int32_t iters, uint32_t seed, uint32_t *out)
{
    const uint32_t a = seed ^ threadIdx.x, b = 0x7fffffffu - blockIdx.x;
    uint32_t acc[CHAINS];
#pragma unroll
    for (int k = 0; k < CHAINS; ++k) acc[k] = threadIdx.x * CHAINS + k;
    for (int32_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < CHAINS; ++k) {
            acc[k] = min(acc[k] + a, b);
            asm volatile("" : "+v"(acc[k]));
        }
    }
    uint32_t r = 0;
#pragma unroll
    for (int k = 0; k < CHAINS; ++k) r ^= acc[k];
    if (r == seed) out[blockIdx.x] = r;  // practically never taken; keeps the chains' work
}

__global__ __launch_bounds__(256) void k_copy(const uint4 *__restrict__ src, uint4 *__restrict__ dst, int64_t n)
{
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += step) dst[i] = src[i];
}

// A streaming read: every lane folds the 16-byte words it loads into one value, written
// only if it equals a value it practically never takes (so the loads stay).
__global__ __launch_bounds__(256) void k_read(const uint4 *__restrict__ src, uint32_t *out, int64_t n)
{
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    uint32_t acc = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += step) {
        const uint4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u) out[blockIdx.x] = acc;
}

// Best of three timed runs of `launch` after one warm-up, in seconds.
template <class F>
int best_of_three(hipStream_t st, F launch, double *sec)
{
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return RKC_E_DEVICE;
    int rc = RKC_OK;
    float best = 1e30f;
    for (int rep = 0; rep < 4 && rc == RKC_OK; ++rep) {
        if (hipEventRecord(e0, st) != hipSuccess) { rc = RKC_E_DEVICE; break; }
        launch();
        if (hipGetLastError() != hipSuccess || hipEventRecord(e1, st) != hipSuccess ||
            hipEventSynchronize(e1) != hipSuccess) { rc = RKC_E_DEVICE; break; }
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) { rc = RKC_E_DEVICE; break; }
        if (rep > 0) best = std::min(best, ms);
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    *sec = best * 1e-3;
    return rc;
}

}  // namespace

extern "C" int rkc_valu_int32_rate(int32_t iters, double *ops_per_s)
{
    if (!ops_per_s || iters < 1 || iters > (1 << 24)) return RKC_E_INVAL;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        return RKC_E_DEVICE;
    const int blocks = cus * 8;
    uint32_t *out = nullptr;
    if (hipMalloc(&out, (size_t)blocks * sizeof(uint32_t)) != hipSuccess) return RKC_E_NOMEM;
    hipStream_t st = nullptr;
    if (hipStreamCreate(&st) != hipSuccess) { (void)hipFree(out); return RKC_E_DEVICE; }
    double sec = 0.0;
    const int rc = best_of_three(st, [&] { hipLaunchKernelGGL(k_valu, dim3(blocks), dim3(256), 0, st, iters, 0x9e3779b9u, out); }, &sec);
    (void)hipStreamDestroy(st);
    (void)hipFree(out);
    if (rc != RKC_OK) return rc;
    *ops_per_s = 2.0 * CHAINS * (double)iters * blocks * 256 / sec;
    return RKC_OK;
}

extern "C" int rkc_copy_bandwidth(int64_t bytes, double *bytes_per_s)
{
    if (!bytes_per_s || bytes <= 0 || bytes % 16 || bytes > (int64_t(1) << 36)) return RKC_E_INVAL;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        return RKC_E_DEVICE;
    void *src = nullptr, *dst = nullptr;
    if (hipMalloc(&src, (size_t)bytes) != hipSuccess) return RKC_E_NOMEM;
    if (hipMalloc(&dst, (size_t)bytes) != hipSuccess) { (void)hipFree(src); return RKC_E_NOMEM; }
    hipStream_t st = nullptr;
    int rc = hipStreamCreate(&st) == hipSuccess && hipMemsetAsync(src, 1, (size_t)bytes, st) == hipSuccess
                 ? RKC_OK
                 : RKC_E_DEVICE;
    // the grid that copies fastest: fewer, longer-running workgroups tend to win
    double sec = 1e30;
    const int64_t n = bytes / 16;
    for (int per_cu : {2, 4, 8, 16}) {
        if (rc != RKC_OK) break;
        double t = 0.0;
        rc = best_of_three(st, [&] {
            hipLaunchKernelGGL(k_copy, dim3(cus * per_cu), dim3(256), 0, st, (const uint4 *)src, (uint4 *)dst, n);
        }, &t);
        sec = std::min(sec, t);
    }
    if (st) (void)hipStreamDestroy(st);
    (void)hipFree(src);
    (void)hipFree(dst);
    if (rc != RKC_OK) return rc;
    *bytes_per_s = 2.0 * (double)bytes / sec;
    return RKC_OK;
}

extern "C" int rkc_read_bandwidth(int64_t bytes, double *bytes_per_s)
{
    if (!bytes_per_s || bytes <= 0 || bytes % 16 || bytes > (int64_t(1) << 36)) return RKC_E_INVAL;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        return RKC_E_DEVICE;
    constexpr int MAX_PER_CU = 16;
    void *src = nullptr;
    uint32_t *out = nullptr;
    if (hipMalloc(&src, (size_t)bytes) != hipSuccess) return RKC_E_NOMEM;
    if (hipMalloc(&out, (size_t)cus * MAX_PER_CU * sizeof(uint32_t)) != hipSuccess) {
        (void)hipFree(src);
        return RKC_E_NOMEM;
    }
    hipStream_t st = nullptr;
    int rc = hipStreamCreate(&st) == hipSuccess && hipMemsetAsync(src, 1, (size_t)bytes, st) == hipSuccess
                 ? RKC_OK
                 : RKC_E_DEVICE;
    double sec = 1e30;
    const int64_t n = bytes / 16;
    for (int per_cu : {2, 4, 8, MAX_PER_CU}) {
        if (rc != RKC_OK) break;
        double t = 0.0;
        rc = best_of_three(st, [&] {
            hipLaunchKernelGGL(k_read, dim3(cus * per_cu), dim3(256), 0, st, (const uint4 *)src, out, n);
        }, &t);
        sec = std::min(sec, t);
    }
    if (st) (void)hipStreamDestroy(st);
    (void)hipFree(src);
    (void)hipFree(out);
    if (rc != RKC_OK) return rc;
    *bytes_per_s = (double)bytes / sec;
    return RKC_OK;
}
