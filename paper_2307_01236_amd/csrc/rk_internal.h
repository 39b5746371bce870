// rk_internal.h -- shared definitions of librkrotor's host code and HIP kernels.
//
// Table layout in HBM (one row per span, diagonal-major):
//   row(s,t) = off(d) + s with d = t - s and off(d) = sum_{d' < d} (L - d'),
//   element (s,t,m) at tab[row(s,t) * stride + m], m in [0, W), W = M + 1,
//   stride = W rounded up to a multiple of 64 int32 (256 B) so every row starts
//   on a 256-byte boundary.
// A span-length diagonal is thus a contiguous slab of (L - d) rows.
//
// Inside the device code "infinity" is DINF = 2^30 - 1: a saturated partial
// sum (at most DINF) plus a table value (at most DINF) still fits in int32, so
// the hot loops need no 64-bit or saturating arithmetic.  Every finite value
// is at most RK_TIME_LIMIT < DINF (checked when the chain is created); the
// host turns DINF into RK_INF on the way out.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "rk.h"

namespace rk {

constexpr int32_t DINF = (1 << 30) - 1;
static_assert(RK_TIME_LIMIT < DINF, "finite values must stay below the device infinity");

// Per-chain arrays derived on the host (App. C quantities), resident on the device.
struct DevChain {
    int32_t L, K;
    const int32_t *x;      // [L+1]  activation sizes
    const int32_t *xbar;   // [L*K]  x_{s+1} + mem_s^o: what F_s^o leaves live
    const int32_t *c1;     // [L*K]  r(F_s^o) + r(B_s^o)
    const int32_t *need1;  // [L*K]  smallest m at which option o of block s is valid
    const int32_t *P;      // [L*L]  P[s*L+i] = sum_{k=s}^{i-1} r(F_k^0)        (i > s)
    const int32_t *need2;  // [L*L]  smallest m at which the sweep s..i-1 is valid (i > s)
};

__host__ __device__ inline int64_t row_of(int32_t L, int32_t s, int32_t t)
{
    const int64_t d = t - s;
    return d * L - d * (d - 1) / 2 + s;
}

inline int64_t n_rows(int32_t L) { return (int64_t)L * (L + 1) / 2; }
inline int32_t row_stride(int32_t W) { return (W + 63) / 64 * 64; }

// Optional per-launch event bracketing of the fill kernels (benchmark timing).
struct Profiler {
    bool on = false;
    hipStream_t stream = nullptr;
    std::vector<hipEvent_t> events;  // pool, 2 per launch
    std::vector<int32_t> kinds;      // kernel kind of each bracketed launch
    int32_t n = 0;                   // launches bracketed in the current solve
    hipError_t before(int32_t kind);
    hipError_t after();
    void reset(hipStream_t s) { stream = s; n = 0; kinds.clear(); }
};

// Kernel kinds of the fill, in the order rk_fill_kernel_stats reports them.
enum FillKernel : int32_t { KFILL_DIAG = 0, KFILL_NKINDS };
extern const char *const kFillKernelNames[KFILL_NKINDS];

// Launchers (rk_kernels.hip).  All return hipError_t of the launch.
hipError_t launch_fill(const DevChain &ch, int32_t *tab, int32_t W, int32_t stride,
                       hipStream_t stream, int32_t *launches, Profiler *prof);
hipError_t launch_arg_row(const DevChain &ch, const int32_t *tab, int32_t W, int32_t stride,
                          int32_t s, int32_t t, int16_t *out, hipStream_t stream);
// Alg. 3 on the device; res[0] = number of steps, res[1] = index of the first
// backward, res[2] = status (0 ok, 1 infeasible cell, 2 inconsistent table,
// 3 stack overflow).
hipError_t launch_backtrace(const DevChain &ch, const int32_t *tab, int32_t stride, int32_t m_top,
                            rk_op *ops, int64_t cap, int64_t *res, hipStream_t stream);

}  // namespace rk
