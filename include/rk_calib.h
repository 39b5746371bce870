/*
 * rk_calib.h -- C ABI of librkcalib, measured ceilings of the GPU the rk-Rotor
 * solver runs on, for pricing its kernels against what the chip sustains next to
 * the nominal peaks.  Not part of the solver; the benchmark calls it.
 *
 * The calls run on the current HIP device, on a stream of their own, and wait
 * for their kernels.  Return 0 on success, -1 (RKC_E_INVAL) for a bad argument,
 * -3 (RKC_E_NOMEM) when device memory cannot be allocated, -4 (RKC_E_DEVICE) for
 * any other HIP error.  Results are host values the caller owns.
 */
#ifndef RK_CALIB_H
#define RK_CALIB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { RKC_OK = 0, RKC_E_INVAL = -1, RKC_E_NOMEM = -3, RKC_E_DEVICE = -4 };

/*
 * Sustained int32 VALU rate: every lane of a full grid (eight workgroups of four
 * wavefronts per compute unit) runs eight independent chains of acc = min(acc + a, b)
 * for `iters` steps -- the add and the min that one relaxation of the recurrence costs
 * (App. C, Eq. fn).  *ops_per_s receives lane operations per second (two per step),
 * the best of three timed launches after one warm-up.  iters must be in [1, 2^24].
 */
int rkc_valu_int32_rate(int32_t iters, double *ops_per_s);

/*
 * Sustained device-memory bandwidth: a copy kernel with 16-byte loads and stores moves
 * `bytes` (a positive multiple of 16, at most 2^36) from one device buffer to another,
 * with 2, 4, 8 and 16 workgroups of 256 lanes per compute unit; *bytes_per_s receives
 * bytes read plus bytes written per second of the fastest (best of three timed copies
 * after one warm-up, per grid).  Allocates the two buffers for the call and frees them.
 */
int rkc_copy_bandwidth(int64_t bytes, double *bytes_per_s);

/*
 * Sustained device-memory read bandwidth: a kernel with 16-byte loads reads `bytes` (a
 * positive multiple of 16, at most 2^36) of one device buffer and writes nothing back,
 * with 2, 4, 8 and 16 workgroups of 256 lanes per compute unit; *bytes_per_s receives
 * bytes read per second of the fastest (best of three timed reads after one warm-up,
 * per grid).  Allocates the buffer for the call and frees it.
 */
int rkc_read_bandwidth(int64_t bytes, double *bytes_per_s);

#ifdef __cplusplus
}
#endif
#endif /* RK_CALIB_H */
