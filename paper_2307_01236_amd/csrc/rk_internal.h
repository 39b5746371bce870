// rk_internal.h -- shared definitions of librkrotor's host code and HIP kernels.
//
// Tables in HBM.  One row per span (s,t), row-major over the upper triangle:
//   row(s,t) = s L - s (s-1)/2 + (t - s),
// so the spans that start at s are consecutive rows (the right operands
// Opt(i, t..t+n) of one split i are n+1 neighbouring rows); one more row
// (index n_rows) holds only "infinity", and SLACK more rows before row 0 and
// after the infinity row keep every operand address a kernel forms in bounds
// (operands that do not exist are read there and then discarded).  A row is
// `stride` int32 wide: `padl` columns of infinity, then the W = M + 1 budget
// columns m = 0..M, then padding to a multiple of 64 (256 B) so every row
// starts 256-byte aligned.
//
//   opt  Opt(s,t,m) at opt[row(s,t)*stride + padl + m].  The left pad lets a
//        read at m - xbar (case 1) run unmasked: columns below 0 read
//        infinity.  Before a span is final its slot holds the partial minimum
//        that the products left there.
//   os   the right operand of Eq. fn, written with Opt when a row becomes final:
//        os[row(i,t)*stride + padl + m] = Opt(i,t,m - x_i) for x_i <= m < W,
//        infinity below x_i, so a split's right operand is read at column m,
//        in step with its left operand and 256-byte aligned like it (read at
//        m - x_i in opt, a wave's 256 bytes straddle three 128-byte lines
//        unless x_i is a multiple of 32).
//   ap   the left operand of Eq. fn, precomputed when a row becomes final:
//        ap[row(s,i-1)*stride + padl + m] = P[s][i] + Opt(s,i-1,m) if the
//        no-save sweep s..i-1 fits in m, else infinity (saturated).
//   hopt, aq  (the saving sweep only) H of case 3 and its left operand, laid out alike.
//
// Inside the device code "infinity" is DINF = 2^30 - 1: ap (at most DINF) plus
// an Opt value (at most DINF) fits in int32, so the hot loops are a plain add
// and a min.  Every finite value is at most RK_TIME_LIMIT < DINF (checked
// when the chain is created); the host turns DINF into RK_INF on the way out.
// The band product adds with unsigned saturation instead: a candidate that is
// not a split of its cell has one operand forced to DINF, and its other operand
// may be any 32-bit pattern (a row not written yet), so the sum stays >= DINF.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "rk.h"

namespace rk {

constexpr int32_t DINF = (1 << 30) - 1;
static_assert(RK_TIME_LIMIT < DINF, "finite values must stay below the device infinity");

// Spans per band: every band of BAND span lengths gets one tiled product over
// the splits whose two operands are older than the band.  Inside a band, mid
// products every MIDMIN spans cover the splits whose longer operand lies in the
// band's earlier part, so that a diagonal's own launch adds fewer than 2 MIDMIN.
// (A level of width 4 saved the finalize more table reads than its 48 launches
// cost only while the finalize read its right operands unaligned and without the
// lower bound; now it costs 0.3 ms on every table size measured.)
constexpr int32_t BAND = 32;
constexpr int32_t MIDMIN = 8;

// Splits per chunk of the band product.
constexpr int32_t PROD_CI = 2;

// The products address an operand block through one buffer descriptor with 32-bit byte
// offsets from its first row.  The widest block spans at most OFFSET_SPAN_L * (L - 1) +
// OFFSET_SPAN_C rows: a width-16 mid tile's group B reads left operands of 18 consecutive
// rows s, each L - 1 - s rows after the previous one (the band product's blocks span at most
// 3 (L - 1) + 2 and L + 41 rows).  A workspace whose span reaches 2 GiB is refused.
constexpr int32_t OFFSET_SPAN_L = 18, OFFSET_SPAN_C = 64;

// Rows of slack before row 0 and after the infinity row of each table.
constexpr int32_t SLACK = 32;

// Per-chain arrays derived on the host (App. C quantities), resident on the device.
struct DevChain {
    int32_t L, K;
    const int32_t *x;      // [L+1]  activation sizes
    const int32_t *xbar;   // [L*K]  x_{s+1} + mem_s^o: what F_s^o leaves live
    const int32_t *c1;     // [L*K]  r(F_s^o) + r(B_s^o)
    const int32_t *need1;  // [L*K]  smallest m at which option o of block s is valid
    const int32_t *need1max;  // [L] max_o need1[s][o]: every option of block s is valid from here
    const int32_t *P;      // [L*L]  P[s*L+i] = sum_{k=s}^{i-1} r(F_k^0)        (i > s)
    const int32_t *need2;  // [L*L]  smallest m at which the sweep s..i-1 is valid (i > s)
    // Where storing everything fits (per span row, row_of order): from budget msa on,
    // Opt(s,t,m) = lb, the sum over the span's blocks of their cheapest r(F)+r(B) (see
    // rk_chain_create).  msa saturates at 2^30 (far beyond any budget column); the host
    // uses it to size each launch.
    const int32_t *lb;     // [L(L+1)/2]
    const int32_t *h_msa;  // [L(L+1)/2], host memory
    // The saving sweep (both null when it is off): c3 = r(F)+r(B)+refwd per option slot
    // [L*K], need3 [L*L] the thresholds of the sweeps of H (the input inside the budget).
    const int32_t *c3;
    const int32_t *need3;
    const int32_t *h_msaH;  // [L(L+1)/2], host memory: from msaH(s,t) on, H(s,t) = lb(s,t) + P[s][s+1]
    int32_t xbar_halo;     // round64(max xbar): how far left case 1 reads from column m
};

// Largest case-1 shift that the finalize stages in LDS (larger ones read global memory).
constexpr int32_t HMAX = 256;

struct Tables {
    int32_t *opt;
    int32_t *ap;
    int32_t *os;  // the right operand table (above)
    // with the saving sweep (else null): H(s,t,u) and its left operand
    // aq[row(s,i-1)*stride + padl + v] = P[s][i] + Opt(s,i-1,v) if the sweep s..i-1 with its
    // input fits v + x_s, else infinity (H reads it at v = u - x_s)
    int32_t *hopt;
    int32_t *aq;
    int32_t W, stride, padl;
    int64_t inf_row;  // index of the all-infinity row (= number of span rows)
    // Profiling mode 2 only (else null).  ctr: the finalize candidates skipped by the lower
    // bound lb(s,t) + P(s,i), zeroed by the fill's first launch (layout: CTR_* below).  rec:
    // one entry per workgroup of the current product or mid launch (tile order of its grid):
    // a band product's first split past the range it relaxed, a mid tile's 1 if it ran and
    // 0 if its lower bound skipped it.
    unsigned long long *ctr;
    int32_t *rec;
};

// The finalize skip counter: a workgroup adds into slot blockIdx.x % CTR_SLOTS, the slots
// CTR_PITCH counters (128 bytes) apart, so that the atomics spread over the L2 channels
// instead of queueing on one address; the host sums the slots.
constexpr int32_t CTR_SLOTS = 256, CTR_PITCH = 16;
constexpr int64_t CTR_WORDS = (int64_t)CTR_SLOTS * CTR_PITCH;

// Rows of one table in the workspace: slack, the span rows, the infinity row, slack.
inline int64_t table_rows(int32_t L) { return (int64_t)L * (L + 1) / 2 + 1 + 2 * SLACK; }

__host__ __device__ inline int64_t row_of(int32_t L, int32_t s, int32_t t)
{
    return (int64_t)s * L - (int64_t)s * (s - 1) / 2 + (t - s);
}

inline int64_t n_rows(int32_t L) { return (int64_t)L * (L + 1) / 2; }
inline int32_t round64(int64_t v) { return (int32_t)((v + 63) / 64 * 64); }

// Optional per-launch event bracketing of the fill kernels (benchmark timing).
struct Profiler {
    bool on = false;
    bool count = false;  // also the device candidate counts (the kernels' counting variants)
    hipStream_t stream = nullptr;
    std::vector<hipEvent_t> events;  // pool, 2 per launch
    std::vector<int32_t> kinds;      // kernel kind of each bracketed launch
    int32_t n = 0;                   // launches bracketed in the current solve
    int64_t work[8] = {};            // relaxations of the recurrence per kernel kind in the current solve
    int64_t eval[8] = {};            // relaxations evaluated (tiles past msa skip); profiling only
    int64_t bytes[8] = {};           // compulsory table traffic of what runs; profiling only
    unsigned long long *d_ctr = nullptr;  // device counters of Tables::ctr (mode 2)
    int32_t *d_rec = nullptr;             // Tables::rec (mode 2), room for rec_cap entries
    int64_t rec_cap = 0;
    std::vector<int32_t> h_rec;           // the last launch's records, read back
    bool ctr_valid = false;               // the last fill counted: d_ctr holds its counts
    // two events from the pool for the next launch, which is of kind `kind`
    hipError_t slot(int32_t kind, hipEvent_t *start, hipEvent_t *stop);
    // mode 2: room for n records of the next launch (waits for the stream before it grows)
    hipError_t records(hipStream_t s, int64_t n);
    // mode 2: the last launch's n records into h_rec (waits for the stream)
    hipError_t read_records(hipStream_t s, int64_t n);
    void reset(hipStream_t s)
    {
        stream = s;
        n = 0;
        kinds.clear();
        for (int64_t &w : work) w = 0;
        for (int64_t &w : eval) w = 0;
        for (int64_t &b : bytes) b = 0;
    }
};

// Kernel kinds of the fill, in the order rk_fill_kernel_stats reports them.
enum FillKernel : int32_t { KFILL_PRODUCT = 0, KFILL_MID, KFILL_FINALIZE, KFILL_INIT, KFILL_NKINDS };
static_assert(KFILL_NKINDS <= 8, "Profiler::work holds 8 kinds");
extern const char *const kFillKernelNames[KFILL_NKINDS];

// Launchers (rk_kernels.hip).  All return hipError_t of the launch.
hipError_t launch_fill(const DevChain &ch, const Tables &tb, hipStream_t stream, int32_t *launches,
                       Profiler *prof);
hipError_t launch_arg_row(const DevChain &ch, const Tables &tb, int32_t s, int32_t t, int16_t *out,
                          hipStream_t stream);
// Alg. 3 on the device; res[0] = number of steps, res[1] = index of the first
// backward, res[2] = status (0 ok, 1 infeasible cell, 2 inconsistent table,
// 3 stack overflow).
hipError_t launch_backtrace(const DevChain &ch, const Tables &tb, int32_t m_top, rk_op *ops,
                            int64_t cap, int64_t *res, hipStream_t stream);

}  // namespace rk
