// rk_kernels.hip -- HIP kernels of librkrotor for gfx950.
//
// The fill evaluates, for every span (s,t) and budget m, Eq. (all) of App. C:
// the minimum of case 1 (Eq. fe: one saving option o of block s, then the
// rest s+1..t with m - xbar) and case 2 (Eq. fn: a no-save sweep s..i-1 that
// keeps x_i, the subproblem i..t with m - x_i, then s..i-1 with m).  Spans of
// one length d = t - s only read shorter spans, so a whole diagonal is one
// data-parallel step over (s, m); lanes run along m, so every table read of a
// wave is one contiguous 256-byte segment (shifted by a per-block constant).
//
// Only values are stored: Opt and ap, the left operand of Eq. fn with the sweep's
// time and validity folded in.  Which choice realises a minimum is recomputed from
// the finished table where it is needed (Alg. 3 does the same: it asks which case
// attains Opt(s,t,m)), so the fill keeps no argmin bookkeeping.
#include "rk_internal.h"

#include <hip/hip_ext.h>

#include <algorithm>
#include <type_traits>

namespace rk {

const char *const kFillKernelNames[KFILL_NKINDS] = {"k_product", "k_mid", "k_finalize", "k_init_inf_rows"};

hipError_t Profiler::slot(int32_t kind, hipEvent_t *start, hipEvent_t *stop)
{
    while ((int32_t)events.size() < 2 * (n + 1)) {
        hipEvent_t e;
        hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) return err;
        events.push_back(e);
    }
    kinds.push_back(kind);
    *start = events[2 * n];
    *stop = events[2 * n + 1];
    ++n;
    return hipSuccess;
}

hipError_t Profiler::records(hipStream_t s, int64_t n)
{
    if (n <= rec_cap) return hipSuccess;
    hipError_t e = hipStreamSynchronize(s);  // the previous launch may still write the old buffer
    if (e != hipSuccess) return e;
    if (d_rec && (e = hipFree(d_rec)) != hipSuccess) return e;
    d_rec = nullptr;
    rec_cap = 0;
    if ((e = hipMalloc(&d_rec, n * sizeof(int32_t))) != hipSuccess) return e;
    rec_cap = n;
    return hipSuccess;
}

hipError_t Profiler::read_records(hipStream_t s, int64_t n)
{
    h_rec.resize(n);
    hipError_t e = hipMemcpyAsync(h_rec.data(), d_rec, n * sizeof(int32_t), hipMemcpyDeviceToHost, s);
    return e != hipSuccess ? e : hipStreamSynchronize(s);
}

// Launch one fill kernel.  With profiling on, the runtime records a pair of events with the
// dispatch itself (hipExtLaunchKernelGGL), at the kernel's start and end, so the elapsed
// time is the kernel's own, without the gaps between launches.
template <typename K, typename... Args>
static hipError_t launch(Profiler *prof, int32_t kind, K kernel, dim3 grid, dim3 block, hipStream_t stream,
                         Args... args)
{
    if (!prof->on) {
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
        return hipGetLastError();
    }
    hipEvent_t e0 = nullptr, e1 = nullptr;
    const hipError_t e = prof->slot(kind, &e0, &e1);
    if (e != hipSuccess) return e;
    hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, e0, e1, 0, args...);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// The all-infinity row and the slack rows of every table (read in place of operands that
// do not exist yet).  Block y picks the row: slack before row 0, or the infinity row and
// the slack after it, of table y / (2 SLACK + 1) (opt, ap, then hopt and aq).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_init_inf_rows(Tables tb)
{
    constexpr int32_t PER_TABLE = 2 * SLACK + 1;
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int32_t y = (int32_t)blockIdx.y, k = y % PER_TABLE, table = y / PER_TABLE;
    const int64_t row = k < SLACK ? (int64_t)k - SLACK : tb.inf_row + (k - SLACK);
    int32_t *const base = table == 0 ? tb.opt : table == 1 ? tb.ap : table == 2 ? tb.os : table == 3 ? tb.hopt : tb.aq;
    if (j < tb.stride) base[row * tb.stride + j] = DINF;
    if (tb.ctr && blockIdx.x == 0 && y == 0)
        for (int32_t k = (int32_t)threadIdx.x; k < CTR_SLOTS; k += 256) tb.ctr[k * CTR_PITCH] = 0;
}

// ---------------------------------------------------------------------------------------
// Raw buffer loads: a descriptor per operand block (its range ends with the table's slack),
// a scalar byte offset per operand row and a fixed per-lane byte offset per column.
// ---------------------------------------------------------------------------------------
__device__ inline __amdgpu_buffer_rsrc_t block_rsrc(const int32_t *base, const int32_t *end)
{
    const int64_t bytes = (const char *)end - (const char *)base;
    const uint32_t n = bytes > 0x7fffffffll ? 0x7fffffffu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)n, 0x00020000);
}

// A lane offset past every descriptor's range (ranges stay below 2 GiB): a load with it
// returns 0 without touching memory.
constexpr uint32_t OOB = 0x80000000u;


// ---------------------------------------------------------------------------------------
// Workgroups of a launch go to the 8 XCDs round-robin (id g to XCD g mod 8), and each XCD
// has its own L2.  Tiles are laid out as column chunks x n_idx tiles per chunk, and XCD x
// (g mod 8) takes the chunks x, x + 8, x + 16, ..., each with its n_idx tiles in order.
// Every XCD then keeps whole column chunks (tiles that share operand rows share its L2, at
// about the same time) and gets chunks from the whole budget range, so work that shrinks
// with the budget column (tiles past the store-everything budget) stays even over the
// XCDs.  Launches hold 8 ceil(n_chunks / 8) n_idx workgroups; *chunk >= n_chunks marks a
// spare one.  Correctness does not depend on the dispatch order.
// ---------------------------------------------------------------------------------------
__device__ inline void chunk_tile(uint32_t g, uint32_t n_idx, int32_t *chunk, int32_t *idx)
{
    const uint32_t j = g / 8;
    // scalars: the division is expanded with vector instructions, and without the hint
    // every address derived from the tile would be computed (and loaded) per lane
    *chunk = __builtin_amdgcn_readfirstlane((int32_t)(g % 8 + 8 * (j / n_idx)));
    *idx = __builtin_amdgcn_readfirstlane((int32_t)(j % n_idx));
}
static inline uint32_t chunk_grid(int32_t n_chunks, int32_t n_idx)
{
    return (uint32_t)(8 * ((n_chunks + 7) / 8) * n_idx);
}

// ---------------------------------------------------------------------------------------
// Band product.  For the spans d in [tau, tau + T) (one band), the part of Eq. fn over
// the splits i whose two operands are older than the band (both s..i-1 and i..t shorter
// than tau).  That is a min-plus product, elementwise in m:
//     acc(s,t) = min_i ap(s,i) + Opt(i, t, m - x_i).
// A workgroup owns 64 consecutive budgets (lane = m) and SW consecutive rows s, in row
// groups of SR rows; each row group's T ends are split over TH waves, so a wave keeps, per
// lane, the SR x TW accumulators of rows s0..s0+SR-1 and ends t = s + tau + kh + k (TW = T/TH
// ends from kh on).  Splits are taken CI at a time.  The right operands
// Opt(i, t, m - x_i) of a chunk, for all NQ ends of the workgroup, are read from the right
// operand table at column m and staged in LDS (each global row read once, then used by up
// to SR waves x rows); each wave reads its own left operands ap(s, i).  The next chunk's operands are loaded into registers while the
// current one is relaxed.
//
// Which candidates are real: split i of cell (s,t) needs s < i <= t and both operand
// spans below tau.  A right operand with span t - i >= tau (this also covers i <= s) is
// replaced by infinity when staged, a left operand with span i - 1 - s >= tau (this also
// covers i > t and splits past the workgroup's range) when used.  Both conditions are
// thresholds in the chunk index, so only the first chunks (right) and the last ones
// (left) mask at all.  Every other candidate that is not a split has one of these infinite
// operands; its other operand is whatever that address holds, and the saturating unsigned
// add keeps the sum at or above DINF.  Cells past the table's last end are computed and
// not stored.  Addresses: one buffer descriptor per chunk and operand table; per split a
// scalar byte offset (advanced incrementally), per row a fixed per-lane offset; all of
// them stay inside the table with its slack rows.
// ---------------------------------------------------------------------------------------
__device__ inline uint32_t sat_add(uint32_t a, uint32_t b) { return __builtin_elementwise_add_sat(a, b); }

// Maximum of a 32-bit value over the 64 lanes of a wavefront (all lanes active): DPP
// exchanges inside each row of 16 lanes, then the four row maxima read as scalars.
__device__ inline uint32_t wave_max_u32(uint32_t v)
{
    v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xb1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
    v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4e, 0xf, 0xf, false));   // quad_perm 2,3,0,1
    v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x124, 0xf, 0xf, false));  // row_ror 4
    v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xf, 0xf, false));  // row_ror 8
    const uint32_t r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return max(max(r0, r1), max(r2, r3));
}

// Splits of the band product's first pass, before it cuts its split range (see k_product).
constexpr int32_t PROD_PREFIX = 40;

// profiling: add v to the counter (one lane per wave calls it)
__device__ inline void count(const Tables &tb, int64_t v)
{
    atomicAdd(&tb.ctr[(int64_t)(blockIdx.x % CTR_SLOTS) * CTR_PITCH], (unsigned long long)v);
}

__device__ inline uint32_t buf_load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff)
{
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0);
}

template <int SR, int TW, int TH, int NW, bool CNT>
__global__ __launch_bounds__(NW * 64) void k_product(DevChain ch, Tables tb, int32_t tau, int32_t n_chunks,
                                                     int32_t n_chunks_h)
{
    // TH waves share SR rows, each keeping TW of the T = TW TH ends of those rows
    constexpr int T = TW * TH, SW = SR * NW / TH, CI = PROD_CI;
    static_assert(NW % TH == 0, "waves split evenly over the ends");
    static_assert(SR - 1 <= OFFSET_SPAN_L && CI - 1 <= OFFSET_SPAN_L, "operand offsets fit the workspace guard");
    constexpr int NQ = (SW + T - 1 + NW - 1) / NW * NW;  // staged ends, padded to the waves
    constexpr int JW = NQ / NW;                           // staged rows per wave and split
    static_assert(CI % 2 == 0, "splits are relaxed in pairs");
    // two staging buffers: chunk c is written to buffer c % 2 while waves that are still
    // relaxing chunk c - 1 read the other one, so one barrier per chunk suffices
    constexpr int QB = CI * NQ * 64;
    __shared__ uint32_t qs[2 * QB];

    const int32_t L = ch.L;
    const uint32_t lane = threadIdx.x & 63;
    // wave index as a scalar: every row choice below is wave-uniform
    const int32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t s_end = L - tau;  // rows that own at least one cell of the band
    const uint32_t n_rb = (uint32_t)(s_end + SW - 1) / SW;
    int32_t chunk, rb;  // row blocks of a column chunk adjacent, chunks spread over the XCDs
    chunk_tile(blockIdx.x, n_rb, &chunk, &rb);
    if (chunk >= n_chunks + n_chunks_h) return;
    // The first n_chunks chunks: case 2 of Opt (left operand ap, partials into opt).  With
    // the saving sweep, n_chunks_h more: H (left operand aq read x_s columns to the left,
    // partials into hopt).  The right operand is Opt in both.
    const bool hp = chunk >= n_chunks;
    if (hp) chunk -= n_chunks;
    const int32_t *const left = hp ? tb.aq : tb.ap;
    int32_t *const out = hp ? tb.hopt : tb.opt;
    const int32_t S0 = rb * SW;
    const uint32_t mchunk = (uint32_t)chunk;
    const int32_t rg = wave / TH, kh = (wave % TH) * TW;  // row group, first end offset
    const int32_t s0 = S0 + rg * SR;
    const int64_t stride = tb.stride;
    const int32_t padl = tb.padl;
    const uint32_t m = mchunk * 64 + lane;
    const uint32_t colb = (uint32_t)(padl + min(m, (uint32_t)tb.W - 1)) * 4u;
    const uint32_t pitch = (uint32_t)stride * 4u;
    const int32_t *const os_end = tb.os + (tb.inf_row + 1 + SLACK) * stride;
    const int32_t *const ap_end = left + (tb.inf_row + 1 + SLACK) * stride;
    const int32_t t0 = S0 + tau;  // first end the workgroup covers
    const int32_t i_lo = S0 + 1, i_hi = min(S0 + SW - 1 + tau, L - 1);


    // right operands: this wave stages ends t0 + wave + NW*jj, which for one split i are
    // rows (i, t0) + wave + NW*jj (the spans starting at i are consecutive rows)
    uint32_t qoff[JW];
#pragma unroll
    for (int jj = 0; jj < JW; ++jj) qoff[jj] = (uint32_t)(jj * NW + wave) * pitch + colb;
    // left operands: row (s0 + r, i - 1) is sum_{s'=s0}^{s0+r-1} (L - 1 - s') rows after (s0, i - 1)
    uint32_t aoff[SR];
    {
        uint32_t delta = 0;
#pragma unroll
        for (int r = 0; r < SR; ++r) {
            // H reads aq(s, i, m - x_s); x_s <= padl unless padl >= W (the read then lands in the pad)
            aoff[r] = delta * pitch + colb - (hp ? 4u * (uint32_t)min(ch.x[min(s0 + r, L)], padl) : 0u);
            delta += (uint32_t)(L - 1 - (s0 + r));
        }
    }

    uint32_t acc[SR][TW];
#pragma unroll
    for (int r = 0; r < SR; ++r)
#pragma unroll
        for (int k = 0; k < TW; ++k) acc[r][k] = DINF;

    // fetch(ic) issues the loads of chunk ic; their values are first used one chunk later
    uint32_t qv[CI][JW], av[CI][SR];
    // Bases of the chunk being fetched: its right-operand block starts one row before
    // (ic, t0), its left-operand block at row (s0, ic - 1).  They advance with ic (row (i+1, t)
    // is L-1-i rows after (i, t), within the workspace guard's 2 GiB) and are recomputed
    // where the chunk order wraps around.
    const int32_t *qcur = nullptr, *acur = nullptr;
    auto seek = [&](int32_t ic) {
        qcur = tb.os + (row_of(L, ic, t0) - 1) * stride;
        acur = left + row_of(L, s0, ic - 1) * stride;
    };
    auto fetch = [&](int32_t ic) {
        // right operands from one row before (ic, t0): split i's rows start rel(i) rows on
        // (the right operand table holds Opt(i, t, m - x_i) at column m)
        const int32_t *const qb = qcur;
        const __amdgpu_buffer_rsrc_t rq = block_rsrc(qb, os_end);
        // Operands that are not used are not read: a staged row whose right span
        // t0 + jj*NW + wave - ic - ii is outside [0, tau), or a left operand whose span
        // ic + ii - 1 - s0 - r is, loads from OOB (value 0; a candidate it takes part in has
        // its other operand masked to infinity, or is itself masked when staged).
        const int32_t qlo = ic - t0 - wave, qhi = ic - S0 - wave;  // kept iff qlo <= jj*NW - ii < qhi
        const bool qall = qlo <= -(CI - 1) && (JW - 1) * NW < qhi;
        uint32_t rel = 1;
#pragma unroll
        for (int ii = 0; ii < CI; ++ii) {
            const int32_t i = ic + ii;
            const uint32_t so = rel * pitch;
            if (qall) {
#pragma unroll
                for (int jj = 0; jj < JW; ++jj) qv[ii][jj] = buf_load(rq, qoff[jj], so);
            } else {
#pragma unroll
                for (int jj = 0; jj < JW; ++jj) {
                    const int32_t e = jj * NW - ii;
                    qv[ii][jj] = buf_load(rq, e >= qlo && e < qhi ? qoff[jj] : OOB, so);
                }
            }
            rel += (uint32_t)max(L - 1 - i, 0);
        }
        // left operands: rows (s0 + r, ic + ii - 1), consecutive in ii
        const int32_t *const ab = acur;
        const __amdgpu_buffer_rsrc_t ra = block_rsrc(ab, ap_end);
        const int32_t a0 = ic - 1 - s0;
        if (a0 - (SR - 1) >= 0 && a0 + CI - 1 < tau) {
#pragma unroll
            for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                for (int r = 0; r < SR; ++r) av[ii][r] = buf_load(ra, aoff[r], (uint32_t)ii * pitch);
        } else {
#pragma unroll
            for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                for (int r = 0; r < SR; ++r) {
                    const int32_t a = a0 + ii - r;
                    av[ii][r] = buf_load(ra, a >= 0 && a < tau ? aoff[r] : OOB, (uint32_t)ii * pitch);
                }
        }
    };

    // Two passes over the splits.  A candidate of split i is at least lb(s,t) + P(s,i):
    // ap(s,i) holds P(s,i) + Opt(s,i-1), and Opt(s,i-1) + Opt(i,t) >= lb(s,i-1) + lb(i,t) =
    // lb(s,t), the sum of the span's cheapest r(F)+r(B) (Opt of any span is at least its lb at
    // every budget); P(s,i) = F(i) - F(s) with F the prefix sums of r(F^0) (row 0 of P) grows
    // with i.  The first pass takes the PROD_PREFIX splits from i_lo on, where every cell's
    // cheapest splits lie; then the workgroup finds the first split i_cut at which
    // F(i) >= acc - lb(s,t) + F(s) for every cell and budget, and the second pass takes only
    // the splits below it: from there on no candidate can lower a partial minimum.
    //
    // Within a pass, neighbouring row blocks share most right operand rows at equal split i,
    // so the row blocks of a group start at one common split (anchor) and wrap around:
    // [anchor, hi] in order, then [lo, anchor).  Their ranges differ by a shift only, so after
    // the wrap they again visit equal i at about equal times, and the rows they share are read
    // from L2 while still there.  (A chunk of the second part may run into the anchor: its
    // splits are relaxed twice, which leaves the minimum unchanged.)
    constexpr int32_t DONE = 0x7fffffff;
    auto pass = [&](int32_t lo, int32_t hi, int32_t anchor) {
        auto next_chunk = [&](int32_t c) {
            if (c >= anchor) return c + CI <= hi ? c + CI : (lo < anchor ? lo : DONE);
            return c + CI < anchor ? c + CI : DONE;
        };
        seek(anchor);
        fetch(anchor);
        for (int32_t ic = anchor, buf = 0; ic != DONE; buf ^= 1) {
            const int32_t inext = next_chunk(ic);
            uint32_t *const qsb = qs + buf * QB;
            const uint32_t *const qw = qsb + (rg * SR + kh) * 64 + lane;
            // staged row jj*NW + wave of split ic + ii is final iff jj*NW - ii < qlim
            const int32_t qlim = ic - S0 - wave;
            if (qlim > (JW - 1) * NW) {
#pragma unroll
                for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                    for (int jj = 0; jj < JW; ++jj) qsb[(ii * NQ + jj * NW + wave) * 64 + lane] = qv[ii][jj];
            } else {
#pragma unroll
                for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                    for (int jj = 0; jj < JW; ++jj)
                        qsb[(ii * NQ + jj * NW + wave) * 64 + lane] = jj * NW - ii < qlim ? qv[ii][jj] : DINF;
            }
            // left operand of row r, split ic + ii is final iff r - ii > alim
            const int32_t alim = ic - s0 - tau - 1;
            uint32_t a[CI][SR];
            if (alim + CI - 1 < 0) {
#pragma unroll
                for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                    for (int r = 0; r < SR; ++r) a[ii][r] = av[ii][r];
            } else {
#pragma unroll
                for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                    for (int r = 0; r < SR; ++r) a[ii][r] = r - ii > alim ? av[ii][r] : DINF;
            }
            __syncthreads();
            if (inext != DONE) {  // in flight while this chunk is relaxed
                if (inext == ic + CI) {
                    int32_t rows = 0;
#pragma unroll
                    for (int ii = 0; ii < CI; ++ii) rows += L - 1 - (ic + ii);
                    qcur = (const int32_t *)((const char *)qcur + (int64_t)rows * pitch);
                    acur = (const int32_t *)((const char *)acur + (int64_t)CI * pitch);
                } else {
                    seek(inext);
                }
                fetch(inext);
            }
            // acc(s0+r, s0+r+tau+k) = min(acc, ap(s0+r, i) + Opt(i, s0+r+tau+k, m - x_i)), two splits per min
#pragma unroll
            for (int ii = 0; ii < CI; ii += 2)
#pragma unroll
                for (int r = 0; r < SR; ++r)
#pragma unroll
                    for (int k = 0; k < TW; ++k)
                        acc[r][k] = min(min(acc[r][k], sat_add(a[ii][r], qw[(ii * NQ + r + k) * 64])),
                                        sat_add(a[ii + 1][r], qw[((ii + 1) * NQ + r + k) * 64]));
            ic = inext;
        }
    };

    const int32_t n_pre = min((i_hi - i_lo) / CI + 1, PROD_PREFIX / CI);  // chunks of the first pass
    int32_t e_last = min(i_hi, i_lo + CI * n_pre - 1);                      // the last split relaxed
    const int32_t lo2 = i_lo + CI * n_pre;                                // the second pass's first split
    // the first pass of the 4 row blocks of 32 rows: all start at the last block's first
    // split, which lies in every one's first pass, and wrap around
    const int32_t hi1 = i_lo + CI * (n_pre - 1);
    int32_t anchor1 = S0 / (4 * SW) * (4 * SW) + 3 * SW + 1;
    if (anchor1 < i_lo || anchor1 > hi1) anchor1 = i_lo;
    pass(i_lo, hi1, anchor1);
    if (lo2 <= i_hi) {
        // the cut: the largest acc - lb(s,t) + F(s) over the wave's real cells and budgets
        // (infinite partials keep every split), then over the workgroup through the staging
        // buffer, which the first pass no longer reads
        uint32_t thr = 0;
#pragma unroll
        for (int r = 0; r < SR; ++r) {
            const int32_t s = s0 + r;
            if (s < s_end) {
                const int32_t *const lbr = ch.lb + row_of(L, s, s + tau + kh);
                const uint32_t fs = (uint32_t)ch.P[s];  // F(s) = P[0][s]
#pragma unroll
                for (int k = 0; k < TW; ++k)
                    if (s + tau + kh + k < L)
                        thr = max(thr, acc[r][k] >= (uint32_t)DINF ? 0xffffffffu : acc[r][k] - (uint32_t)lbr[k] + fs);
            }
        }
        if (m >= (uint32_t)tb.W) thr = 0;
        thr = wave_max_u32(thr);
        __syncthreads();  // every wave is done with the staging buffers
        if (lane == 0) qs[wave] = thr;
        __syncthreads();
#pragma unroll
        for (int w = 0; w < NW; ++w) thr = max(thr, qs[w]);
        thr = __builtin_amdgcn_readfirstlane(thr);
        // i_cut: the first split i in [lo2, i_hi + 1) with F(i) >= thr (F is non-decreasing)
        int32_t cl = lo2, ch_ = i_hi + 1;
        if (thr != 0xffffffffu) {
            while (cl < ch_) {
                const int32_t mid = (cl + ch_) >> 1;
                if ((uint32_t)ch.P[mid] >= thr) ch_ = mid;
                else cl = mid + 1;
            }
        }
        const int32_t hi2 = thr == 0xffffffffu ? i_hi : cl - 1;
        if (lo2 <= hi2) {
            // the second pass of a group of n2 row blocks starts at the last block's first
            // split lo2, which lies in every block's uncut range [lo2, i_hi]; a block whose
            // cut falls below it starts at its own lo2
            const int32_t n2 = max(1, (tau - PROD_PREFIX - 2) / SW + 2);
            int32_t anchor = rb / n2 * n2 * SW + (n2 - 1) * SW + 1 + CI * n_pre;
            if (anchor > hi2 || anchor < lo2) anchor = lo2;
            __syncthreads();  // the staging buffer held the thresholds
            pass(lo2, hi2, anchor);
            e_last = min(i_hi, anchor + CI * ((hi2 - anchor) / CI) + CI - 1);
        }
    }
    if (CNT && threadIdx.x == 0)  // profiling: every cell of the tile relaxed its splits i <= e_last
        tb.rec[(int64_t)(hp ? n_chunks + chunk : chunk) * n_rb + rb] = e_last + 1;
    if (m >= (uint32_t)tb.W) return;
    // the wave's ends t0r..t0r+TW-1 of row s are consecutive rows: one descriptor per row s
    // covers those inside the table, and a store past them is dropped by its range check
    const uint32_t cst = (uint32_t)(padl + m) * 4u;
#pragma unroll
    for (int r = 0; r < SR; ++r) {
        const int32_t s = s0 + r, t0r = s + tau + kh;
        if (s >= s_end || t0r >= L) continue;
        const int32_t nk = min(TW, L - t0r);
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            out + row_of(L, s, t0r) * stride, (short)0, (int)(nk * pitch), 0x00020000);
#pragma unroll
        for (int k = 0; k < TW; ++k)
            __builtin_amdgcn_raw_buffer_store_b32((int32_t)acc[r][k], rs, (int)(cst + (uint32_t)k * pitch), 0, 0);
    }
}

// ---------------------------------------------------------------------------------------
// Mid product of width WD inside a band.  For the spans d in [tau, tau + WD), lo = tau - WD,
// the part of Eq. fn over the splits whose longer operand has a span in [lo, tau):
//   group A: left span a = i-1-s in [lo, tau) (the right span d-1-a is then below 2 WD - 1)
//   group B: right span b = t-i in [lo, tau) (the left span is then below 2 WD - 1)
// Every lo > 0 used is at least 2 WD, so the groups are disjoint and their short operand
// spans lie below lo.  With lo == 0 the launch covers the splits whose two spans are both
// below WD (group A with the right span bounded too).  These are splits that one finalize
// launch per diagonal would otherwise read operand by operand.
// Both groups write every cell of the spans; each folds into the stored partial with an
// atomic minimum, so they run in one launch in any order.
// A wave owns R = 4 rows (group A: rows s0 + r, ends s0 + r + tau + k) or R ends (group B:
// ends t0 + r, rows t0 + r - tau - k), k < WD, and 64 budgets.  The tile's WD + R - 1
// splits are unrolled; which (split, row) pairs are real depends only on their positions
// in the tile, so it is known at compile time and nothing is masked.  A split's operand
// loads are issued one split ahead of its relaxation.  Cells past the table are computed
// and not stored (their operand rows are clamped into the table).
// ---------------------------------------------------------------------------------------
// Calls f(integral_constant<int, U>) for U = B .. E-1 in order: a loop unrolled by
// construction, whose index is a compile-time constant in the body.
template <int B, int E, typename F>
__device__ inline void static_for(F &&f)
{
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// rows (group A) or ends (group B) of a mid product tile
template <int WD>
constexpr int mid_rows() { return 4; }

// load at a byte offset from a wave-uniform base (one scalar base + one 32-bit lane offset)
__device__ inline int32_t ldb(const int32_t *base, uint32_t byte_off)
{
    return *(const int32_t *)((const char *)base + byte_off);
}

// Returns false when the tile is skipped by its lower bound.  Always inlined: k_mid calls it
// from three places, and an outlined call would need a scratch frame.
template <int WD, bool GA, bool LO0>
__device__ __attribute__((always_inline)) inline bool mid_tile(const DevChain &ch, const Tables &tb, int32_t tau, int32_t accumulate,
                                int32_t g, bool hp)
{
    constexpr int R = mid_rows<WD>(), NS = WD + R - 1, NJ = R + WD - 1;
    static_assert(WD == 4 || WD == 8 || WD == 16, "widths 4, 8 and 16");
    static_assert(GA || !LO0, "lo == 0 is group A only");
    static_assert(NJ - 1 <= OFFSET_SPAN_L && NJ + 1 <= OFFSET_SPAN_C, "operand offsets fit the workspace guard");
    const int32_t L = ch.L, W = tb.W, lo = tau - WD;
    const int32_t lane = (int32_t)(threadIdx.x & 63);
    const int32_t n_blk = (L - tau + R - 1) / R;  // row blocks (A), end blocks (B)
    const int32_t mc = g / n_blk, blk = g % n_blk;
    const int64_t stride = tb.stride;
    const uint32_t pitch = (uint32_t)stride * 4u;
    const int32_t padl = tb.padl;
    const int32_t m = mc * 64 + lane;
    const uint32_t col = (uint32_t)(padl + min(m, W - 1)) * 4u;
    const int32_t *const os_end = tb.os + (tb.inf_row + 1 + SLACK) * stride;
    // case 2 of Opt (left ap, into opt) or, with hp, H of the saving sweep (left aq read x_s
    // columns to the left, into hopt); the right operand Opt(i, t, m - x_i) from the right
    // operand table at column m
    const int32_t *const left = hp ? tb.aq : tb.ap;
    int32_t *const out = hp ? tb.hopt : tb.opt;
    const int32_t *const ap_end = left + (tb.inf_row + 1 + SLACK) * stride;
    auto lsh = [&](int32_t srow) { return hp ? 4u * (uint32_t)min(ch.x[min(srow, L)], padl) : 0u; };
    auto rows_between = [&](int32_t s_from, int32_t s_to) {  // row(s_to, t) - row(s_from, t)
        return (int64_t)(s_to - s_from) * (L - 1) - ((int64_t)s_to * (s_to - 1) - (int64_t)s_from * (s_from - 1)) / 2;
    };

    uint32_t acc[R][WD];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int k = 0; k < WD; ++k) acc[r][k] = DINF;

    // Operand r of a split: group A the left operand of row s0 + r, group B the right
    // operand of end t0 + r.  Operand j: group A the right operand of end s0 + tau + j,
    // group B the left operand of row t0 - tau - WD + 1 + j (rows below 0 clamped to 0).
    uint32_t xoff[NJ], roff[R];
    const int32_t base = blk * R;                     // s0 (A) or t0 - tau (B)
    const int32_t i0 = GA ? base + lo + 1 : base + 1;  // the tile's first split
    const int32_t sa = GA ? base : max(base - WD + 1, 0);  // first ap row's start
    if (GA) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) xoff[j] = (uint32_t)j * pitch + col;
#pragma unroll
        for (int r = 0; r < R; ++r)
            roff[r] = (uint32_t)rows_between(base, min(base + r, L - 1)) * pitch + col - lsh(base + r);
    } else {
        const int32_t sb = base - WD + 1;
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            xoff[j] = (uint32_t)rows_between(sa, max(sb + j, 0)) * pitch + col - lsh(max(sb + j, 0));
#pragma unroll
        for (int r = 0; r < R; ++r) roff[r] = (uint32_t)r * pitch + col;
    }

    // Group A (lo > 0): every candidate of row s is at least lb(s,t) + P(s, s+lo+1).  A
    // candidate of split i is ap(s,i) + Opt(i,t), ap(s,i) = P(s,i) + Opt(s,i-1), and
    // Opt(s,i-1) + Opt(i,t) >= lb(s,i-1) + lb(i,t) = lb(s,t), the sum of the span's cheapest
    // r(F)+r(B) (Opt of any span is at least its lb at every budget); P(s,i) grows with i and
    // the tile's splits of row s start at s + lo + 1.  (With the saving sweep, H's candidates
    // obey the same bound: aq holds the same P.)  When the stored partial of every cell and
    // budget of the tile is already at most that bound, no candidate of the tile can lower
    // it, and the tile is skipped.  The partial then holds the band product's and the wider
    // mids' candidates, which at large spans already make the bound tight: long left spans
    // cost a long recomputation sweep.  (A group B tile folding into the same cells at the
    // same time only lowers the partial; any value it held bounds the final minimum.)
    //
    // The partials are loaded here and tested after the first split's operand loads have
    // been issued, so a tile that is not skipped does not wait for the test.
    constexpr bool TEST = GA && !LO0;
    int32_t pv[TEST ? R : 1][TEST ? WD : 1];
    if constexpr (TEST) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int32_t s = min(base + r, L - tau - 1);
            const int32_t *const pr = out + row_of(L, s, s + tau) * stride;
#pragma unroll
            for (int k = 0; k < WD; ++k)
                pv[r][k] = base + r < L - tau && s + tau + k < L ? ldb(pr + (int64_t)k * stride, col) : -DINF;
        }
    }
    auto skip = [&]() {
        int32_t v = -DINF;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int32_t s = base + r;
            if (s < L - tau) {
                const int32_t pm = ch.P[(int64_t)s * L + s + lo + 1];
                const int32_t *const lbr = ch.lb + row_of(L, s, s + tau);
#pragma unroll
                for (int k = 0; k < WD; ++k)
                    if (s + tau + k < L) v = max(v, pv[r][k] - lbr[k] - pm);
            }
        }
        if (m >= W) v = -DINF;
        return (int32_t)wave_max_u32((uint32_t)(v + DINF)) <= DINF;
    };

    uint32_t vr[2][R], vj[2][NJ];
    // Split u (i = i0 + u) is real for operand r in [u - WD + 1, u]; operand j is needed in
    // [rlo, rhi + WD - 1].  Splits past L - 1 only serve cells past the table (clamped).
    auto load = [&](auto uc, auto bc) {
        constexpr int u = decltype(uc)::value, b = decltype(bc)::value;
        constexpr int rlo = u - WD + 1 > 0 ? u - WD + 1 : 0, rhi = u < R - 1 ? u : R - 1;
        constexpr int jhi = LO0 ? (rhi + WD - 1 < u ? rhi + WD - 1 : u) : rhi + WD - 1;
        const int32_t i = min(i0 + u, L - 1);
        const __amdgpu_buffer_rsrc_t dq = block_rsrc(tb.os + row_of(L, i, base + tau) * stride, os_end);
        const __amdgpu_buffer_rsrc_t da = block_rsrc(left + row_of(L, sa, i0 + u - 1) * stride, ap_end);
#pragma unroll
        for (int r = rlo; r <= rhi; ++r) vr[b][r] = buf_load(GA ? da : dq, roff[r], 0);
#pragma unroll
        for (int j = rlo; j <= jhi; ++j) vj[b][j] = buf_load(GA ? dq : da, xoff[j], 0);
    };
    auto relax = [&](auto uc, auto bc) {
        constexpr int u = decltype(uc)::value, b = decltype(bc)::value;
        constexpr int rlo = u - WD + 1 > 0 ? u - WD + 1 : 0, rhi = u < R - 1 ? u : R - 1;
#pragma unroll
        for (int r = rlo; r <= rhi; ++r)
#pragma unroll
            for (int k = 0; k < WD; ++k) {
                if (GA) {
                    if (!LO0 || r + k <= u)  // with lo == 0 the right span stays below WD
                        acc[r][k] = min(acc[r][k], sat_add(vr[b][r], vj[b][r + k]));
                } else {
                    acc[r][k] = min(acc[r][k], sat_add(vj[b][r - k + WD - 1], vr[b][r]));
                }
            }
    };
    // The splits in the order u = (p + DL) mod NS, p = 0, 1, ...: the tiles of a group (G
    // consecutive tiles, R rows or ends apart; tile g is member w = g mod G) rotate by
    // R (G - 1 - w) so that they all start at the same split i; their ranges differ by a shift only, so they keep visiting
    // equal splits together (also after the wrap) and share their operand rows in L2.
    auto run = [&](auto dc) {
        constexpr int DL = decltype(dc)::value;
        load(std::integral_constant<int, DL % NS>{}, std::integral_constant<int, 0>{});
        if constexpr (TEST)
            if (skip()) return false;
        static_for<0, NS>([&](auto pc) {
            constexpr int p = decltype(pc)::value;
            if constexpr (p + 1 < NS)
                load(std::integral_constant<int, (p + 1 + DL) % NS>{}, std::integral_constant<int, (p + 1) & 1>{});
            relax(std::integral_constant<int, (p + DL) % NS>{}, std::integral_constant<int, p & 1>{});
            // the accumulators are final for this split here, and nothing moves across: only
            // one split's operands are held in registers ahead of their use
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if constexpr (WD == 16)
                    asm volatile("" ::"v"(acc[r][0]), "v"(acc[r][1]), "v"(acc[r][2]), "v"(acc[r][3]),
                                 "v"(acc[r][4]), "v"(acc[r][5]), "v"(acc[r][6]), "v"(acc[r][7]), "v"(acc[r][8]),
                                 "v"(acc[r][9]), "v"(acc[r][10]), "v"(acc[r][11]), "v"(acc[r][12]),
                                 "v"(acc[r][13]), "v"(acc[r][14]), "v"(acc[r][15]));
                else if constexpr (WD == 8)
                    asm volatile("" ::"v"(acc[r][0]), "v"(acc[r][1]), "v"(acc[r][2]), "v"(acc[r][3]),
                                 "v"(acc[r][4]), "v"(acc[r][5]), "v"(acc[r][6]), "v"(acc[r][7]));
                else
                    asm volatile("" ::"v"(acc[r][0]), "v"(acc[r][1]), "v"(acc[r][2]), "v"(acc[r][3]));
            }
            __builtin_amdgcn_sched_barrier(0);
        });
        return true;
    };
    constexpr int G = WD == 16 ? 4 : 2;  // tiles whose split ranges all share a split
    static_assert(R * (G - 1) < NS, "a group's ranges overlap");
    const int32_t wg = g % G;
    bool ran;
    if constexpr (G == 4) {
        if (wg == 0) ran = run(std::integral_constant<int, 3 * R>{});
        else if (wg == 1) ran = run(std::integral_constant<int, 2 * R>{});
        else if (wg == 2) ran = run(std::integral_constant<int, R>{});
        else ran = run(std::integral_constant<int, 0>{});
    } else {
        if (wg == 0) ran = run(std::integral_constant<int, R>{});
        else ran = run(std::integral_constant<int, 0>{});
    }
    if (!ran) return false;

    // store (or fold into the stored partial) through one descriptor per row r: group A
    // cell (s0+r, s0+r+tau+k) is k rows after (s0+r, s0+r+tau); group B cell
    // (t0+r-tau-k, t0+r) is sum_{s'=t0+r-tau-k}^{t0+r-tau-1} (L-1-s') rows before (t0+r-tau, t0+r)
    if (m >= W) return true;
    const uint32_t cst = (uint32_t)(padl + m) * 4u;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int32_t sr = base + r;  // group A: the row; group B: the row of span tau at end t0 + r
        const int32_t tr = base + r + tau;
        if (sr < L - tau) {  // some cell of this row (A) or end (B) lies in the table
            int32_t *const rb = out + row_of(L, sr, tr) * stride;
            int64_t back = 0;  // group B: rows from (sr - k, tr) to (sr, tr)
#pragma unroll
            for (int k = 0; k < WD; ++k) {
                if (!GA && k > 0) back += L - 1 - (sr - k);
                if (GA ? tr + k < L : sr - k >= 0) {
                    int32_t *const p = GA ? rb + (int64_t)k * stride : rb - back * stride;
                    const int32_t v = (int32_t)acc[r][k];
                    if (accumulate) {  // fold into the stored partial in L2, no read-back
                        (void)__hip_atomic_fetch_min((int32_t *)((char *)p + cst), v, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
                    } else {
                        const __amdgpu_buffer_rsrc_t dr =
                            __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)pitch, 0x00020000);
                        __builtin_amdgcn_raw_buffer_store_b32(v, dr, (int)cst, 0, 0);
                    }
                }
            }
        }
    }
    return true;
}

// One launch per level, one wavefront per workgroup and tile (single waves measured a
// little faster than four-wave groups).  Groups A and B fold into the partials with atomic
// min, so they need no order; with lo == 0 only group A, which stores.  Tiles go column
// chunk by column chunk (group A's row blocks, then group B's), and consecutive tiles run
// on one XCD: each XCD keeps the same range of columns as in the finalize launches, whose
// recent rows the mids read.
// The arguments before ch are preloaded into SGPRs when a wave starts, as for the finalize:
// the table pointers and the scalars that the tile's first loads need (tau in bits 0..10 of
// tpack, the fold flag in bit 11; n_tot = n_chunks plus H's chunks).  They stand in for the
// same fields of ch and tb (fill 9.92 -> 9.90 ms).
template <int WD, bool LO0, bool CNT>
__global__ __launch_bounds__(64) void k_mid(int32_t *p_opt, int32_t *p_os, int32_t *p_ap, int32_t stride32,
                                            int32_t padl, int32_t W, int32_t L, int32_t inf_row, uint32_t tpack,
                                            int32_t n_tot, int32_t n_chunks, DevChain ch, Tables tb,
                                            int32_t n_chunks_h)
{
    const int32_t tau = (int32_t)(tpack & 0x7ffu), accumulate = (int32_t)(tpack >> 11);
    tb.opt = p_opt;
    tb.os = p_os;
    tb.ap = p_ap;
    tb.stride = stride32;
    tb.padl = padl;
    tb.W = W;
    tb.inf_row = inf_row;
    ch.L = L;
    constexpr int R = mid_rows<WD>();
    const int32_t n_blk = (ch.L - tau + R - 1) / R;
    // per column chunk: group A's n_blk tiles, then group B's (lo > 0); gi indexes the group.
    // Chunks from n_chunks on are H's (the saving sweep).
    int32_t mc, rem;
    chunk_tile(blockIdx.x, (LO0 ? 1 : 2) * n_blk, &mc, &rem);
    if (mc >= n_tot) return;
    const bool hp = mc >= n_chunks;
    if (hp) mc -= n_chunks;
    const int32_t gi = mc * n_blk + rem % n_blk;
    bool ran;
    if (LO0) ran = mid_tile<WD, true, LO0>(ch, tb, tau, accumulate, gi, hp);
    else if (rem < n_blk) ran = mid_tile<WD, true, false>(ch, tb, tau, accumulate, gi, hp);
    else ran = mid_tile<WD, false, false>(ch, tb, tau, accumulate, gi, hp);
    // profiling: whether the tile ran or its lower bound skipped it
    if (CNT && threadIdx.x == 0) tb.rec[(int64_t)(hp ? n_chunks + mc : mc) * ((LO0 ? 1 : 2) * n_blk) + rem] = ran;
}

// ---------------------------------------------------------------------------------------
// Finalize one span-length diagonal d: cell (s, s+d), budgets m.  Adds to the products'
// partial minimum the splits they did not cover (max(i-1-s, t-i) >= D, D = d rounded down
// to a multiple of midmin, the narrowest mid width) and case 1 (Eq. fe), clamps, writes Opt
// and the row's left operand ap(s, t+1) for the spans that will split after t.
// A workgroup is one wavefront covering FC = 128 budgets of one cell: lane l the columns
// mbase + l and mbase + l + 64, so every scalar address serves two coalesced loads (single
// waves of 128 columns beat four-wave groups of 512 and single waves of 64 or 256).
// Splits go in batches of FB with all loads of a batch issued before any is used; the row
// pointers of a split range advance incrementally.  Case 1 reads one row, Opt(s+1, t, .),
// at K shifts: the wave stages the columns it needs in LDS once (when the largest shift is
// at most HMAX), loading them together with the first splits.
// ---------------------------------------------------------------------------------------
constexpr int32_t FC = 128, FT = 64;  // budgets and threads per workgroup


// the same through a buffer descriptor of one row (bytes [0, pitch) from base): the lane
// offset goes to the load unchanged, with no per-lane address arithmetic
__device__ inline int32_t ldrow(const int32_t *base, uint32_t pitch, uint32_t byte_off)
{
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)pitch, 0x00020000);
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, 0);
}

// A store marked nontemporal: its line is the first the caches let go.  The finalize writes
// several rows per cell that only later launches read, most of them on other XCDs; with
// these stores so marked the fill measured 0.13 ms faster (0.33 ms with the saving sweep),
// the products and mids included, which keep more of their operands in L2.
__device__ inline void st_nt(int32_t v, int32_t *p) { __builtin_nontemporal_store(v, p); }

// The arguments before the first aggregate are preloaded into SGPRs when a wave starts (the
// library is built with kernarg preloading of up to 14 dwords): the three table pointers and
// the scalars that the first table loads depend on, so that a wave issues those loads without
// waiting on a kernel-argument load first (fill 10.37 -> 10.17 ms, 384 launches).  dpack
// holds d, D = d rounded down to a multiple of the narrowest mid width (bits 11..21), whether
// the chain has the saving sweep (bit 22) and the case-1 halo min(xbar_halo, 511) (bits
// 23..31); n_tot = n_chunks plus H's chunks.  The other operands come from ch and tb.
static_assert(RK_MAX_L < 2048, "span lengths are packed in 11 bits");
template <bool CNT>
__global__ __launch_bounds__(FT) void k_finalize(int32_t *p_opt, int32_t *p_os, int32_t *p_ap, uint32_t dpack,
                                                 int32_t n_tot, int32_t n_chunks, int32_t n_run, int32_t L,
                                                 int32_t W, int32_t padl, int32_t stride32, DevChain ch,
                                                 Tables tb, int32_t n_run_h)
{
    constexpr int32_t FB = 8, NC = FC / FT, NST = (HMAX + FC) / FT;
    __shared__ int32_t seg[HMAX + FC], seg3[HMAX + FC];
    const int32_t K = ch.K;
    const int32_t d = (int32_t)(dpack & 0x7ffu);
    const int32_t D = (int32_t)((dpack >> 11) & 0x7ffu);  // the products cover splits with max(a, b) < D
    // Tiles of one column chunk are adjacent in row s, and adjacent tiles run on one XCD: the
    // case-1 row (s+1, t) of a cell was written in the previous launch by the workgroup of
    // the neighbouring tile, so it is often still in that XCD's L2 (rows adjacent: 5.95 ms a
    // fill, column chunks adjacent: 6.15 ms, no XCD-aware order: 6.7 ms).
    int32_t chunk, s;
    chunk_tile(blockIdx.x, (uint32_t)(L - d), &chunk, &s);
    if (chunk >= n_tot) return;
    // chunks from n_chunks on finish H(s, t) of the saving sweep instead of Opt(s, t)
    const bool hp = chunk >= n_chunks;
    if (hp) chunk -= n_chunks;
    const int32_t t = s + d;
    const int32_t mbase = chunk * FC;
    const int32_t lane = (int32_t)(threadIdx.x & 63);
    const int32_t wave = __builtin_amdgcn_readfirstlane((int32_t)(threadIdx.x >> 6));
    const int32_t m0 = mbase + 64 * NC * wave;  // the wave's first column
    const int32_t ml = m0 + lane;           // column c of the lane: ml + 64 c
    const int64_t stride = stride32;
    const uint32_t pitch = (uint32_t)stride * 4u;
    const int64_t row_st = row_of(L, s, t);
    int32_t *const orow = p_opt + row_st * stride + padl;  // column 0
    const int32_t ip = t + 1 < L ? s * L + t + 1 : 0;
    // per-lane column offsets (past the last budget: the last one, computed and not stored)
    uint32_t col[NC];  // byte offsets
#pragma unroll
    for (int c = 0; c < NC; ++c) col[c] = (uint32_t)min(ml + 64 * c, W - 1) * 4u;

    // splits i0 .. i0+n-1: left(s, i-1) + Opt(i, t, m - x_i), left = ap (Opt) or aq read lsh
    // columns to the left (H), the right operand from the right operand table at column m.
    // Pointers at column 0: row (s, i-1) is i-1-s rows after (s, s); row (i+1, t) is L-1-i
    // rows after (i, t)
    int32_t best[NC];
    auto splits = [&](const int32_t *ltab, int32_t lsh, int32_t i0, int32_t n) {
        const int32_t *pa = ltab + (row_of(L, s, s) + (i0 - 1 - s)) * stride + padl - lsh;
        const int32_t *pq = p_os + row_of(L, i0, t) * stride + padl;
        int32_t i = i0;
        for (int32_t j0 = 0; j0 < n; j0 += FB) {
            int32_t va[FB][NC], vq[FB][NC];
#pragma unroll
            for (int u = 0; u < FB; ++u) {
                if (j0 + u < n) {
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        va[u][c] = ldrow(pa, pitch, col[c]);
                        vq[u][c] = ldrow(pq, pitch, col[c]);
                    }
                    pa += stride;
                    pq += (int64_t)(L - 1 - i) * stride;
                    ++i;
                } else {
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        va[u][c] = DINF;
                        vq[u][c] = 0;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < FB; ++u)
#pragma unroll
                for (int c = 0; c < NC; ++c) best[c] = min(best[c], va[u][c] + vq[u][c]);
        }
    };
    // the near splits with a short left span (all of them when D == 0): t - i >= D
    auto near_first = [&](const int32_t *ltab, int32_t lsh) { splits(ltab, lsh, s + 1, D == 0 ? d : d - D); };
    // and those with a long left span, i - 1 - s >= D.  Each of their candidates is at least
    // lb(s,t) + P(s, s+D+1) (ap(s,i) holds P(s,i) + Opt(s,i-1), Opt(s,i-1) + Opt(i,t) >= lb(s,t),
    // and P grows with i; H's aq holds the same P): where the minimum so far is already at most
    // that at every budget of the wave, they are skipped.
    auto near_second = [&](const int32_t *ltab, int32_t lsh) {
        if (D == 0 || d == D) return;
        const int32_t bound = ch.lb[row_st] + ch.P[(int64_t)s * L + s + D + 1];
        uint32_t over = 0;  // some lane's minimum is above the bound
#pragma unroll
        for (int c = 0; c < NC; ++c) over |= (uint32_t)(ml + 64 * c < W && best[c] > bound);
        if (wave_max_u32(over)) splits(ltab, lsh, s + D + 1, d - D);
        else if (CNT && lane == 0)  // profiling: the skipped candidates
            count(tb, (int64_t)(d - D) * min(FC, W - mbase));
    };

    // Opt's second range, in two steps: the test right after the first range (a weaker bound
    // than after case 1, so the range runs a little more often) and, where it does not rule
    // the range out, its loads (d - D < FB splits, one batch), issued before case 1 so that
    // they are in flight while case 1 reads LDS; the minimum is taken after case 1 (fill
    // 10.0 -> 9.9 ms).
    static_assert(MIDMIN <= FB + 1, "the second near range is one batch");
    int32_t va2[FB][NC], vq2[FB][NC];
    auto near_second_issue = [&]() -> bool {
        if (D == 0 || d == D) return false;
        const int32_t bound = ch.lb[row_st] + ch.P[(int64_t)s * L + s + D + 1];
        uint32_t over = 0;
#pragma unroll
        for (int c = 0; c < NC; ++c) over |= (uint32_t)(ml + 64 * c < W && best[c] > bound);
        if (!wave_max_u32(over)) {
            if (CNT && lane == 0) count(tb, (int64_t)(d - D) * min(FC, W - mbase));
            return false;
        }
        const int32_t *pa = p_ap + (row_of(L, s, s) + D) * stride + padl;
        const int32_t *pq = p_os + row_of(L, s + D + 1, t) * stride + padl;
        int32_t i = s + D + 1;
#pragma unroll
        for (int u = 0; u < FB; ++u) {
            if (u < d - D) {
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    va2[u][c] = ldrow(pa, pitch, col[c]);
                    vq2[u][c] = ldrow(pq, pitch, col[c]);
                }
                pa += stride;
                pq += (int64_t)(L - 1 - i) * stride;
                ++i;
            } else {
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    va2[u][c] = DINF;
                    vq2[u][c] = 0;
                }
            }
        }
        return true;
    };

    // From budget msa(s,t) on, storing everything fits and Opt(s,t,m) = lb(s,t).  Chunks from
    // n_run on lie past the msa of every cell of the diagonal (the host's bound): they only
    // store.  The products and mids of these spans ran on at least the chunks below n_run.
    // (The stores stay after every load on every path, so the loads of the per-block and
    // per-option arrays may use the scalar cache.)
    // Opt below msa (the main path): the case-1 row Opt(s+1, t), staged (column mbase - H + q
    // at seg[q]), the products' partial and the first near range are loaded first, before
    // anything that waits on a kernel-argument load: their addresses need only the preloaded
    // arguments.  Opt's paths come first for the same reason.
    const bool main_path = !hp && chunk < n_run;
    const int32_t H = (int32_t)(dpack >> 23);
    const bool staged = main_path && d > 0 && H <= HMAX;
    int32_t stv[NST];
    if (staged) {
        const int32_t *const rrow = p_opt + row_of(L, s + 1, t) * stride;  // column -padl
#pragma unroll
        for (int k = 0; k < NST; ++k) {
            const int32_t q = (int32_t)threadIdx.x + FT * k, c = mbase - H + q;
            // columns left of the row's pad are set to infinity when the row is staged
            stv[k] = ldrow(rrow, pitch, q < H + FC && c >= -padl ? (uint32_t)(c + padl) * 4u : OOB);
        }
    }
    if (main_path) {
#pragma unroll
        for (int c = 0; c < NC; ++c) best[c] = D > 0 ? ldb(orow, col[c]) : DINF;
        near_first(p_ap, 0);
    }
    if (!hp && chunk >= n_run) {
        const int32_t lbv = ch.lb[row_st];
#pragma unroll
        for (int c = 0; c < NC; ++c) best[c] = lbv;
    } else if (!hp) {
        const bool run2 = near_second_issue();
        // with the saving sweep, the row H(s+1, t) of case 3, staged the same way (seg3)
        const bool sweep = (dpack >> 22 & 1u) && d >= 2;
        const int32_t *const rest = d > 0 ? p_opt + row_of(L, s + 1, t) * stride + padl : nullptr;
        const int32_t *const hrest = sweep ? tb.hopt + row_of(L, s + 1, t) * stride + padl : nullptr;
        int32_t stv3[NST];
        if (staged && sweep) {
#pragma unroll
            for (int k = 0; k < NST; ++k) {
                const int32_t q = (int32_t)threadIdx.x + FT * k, c = mbase - H + q;
                // H is read at m - mem >= 0 only (need1 >= mem): columns below 0 are never used
                stv3[k] = q < H + FC && c >= 0 ? hrest[c] : DINF;
            }
        }

        // case 1, option o: r(F_s^o) + r(B_s^o) + Opt(s+1,t,m-xbar), valid iff m >= need1[s][o];
        // case 3 (the saving sweep), option o: r(F)+r(B)+refwd + H(s+1,t,m-mem), same validity
        const int32_t *const c1 = ch.c1 + s * K, *const need1 = ch.need1 + s * K, *const xbar = ch.xbar + s * K;
        const int32_t *const c3 = sweep ? ch.c3 + s * K : nullptr;
        const int32_t x1 = ch.x[s + 1];
        if (d == 0) {
            for (int32_t o = 0; o < K; ++o)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    if (ml + 64 * c >= need1[o]) best[c] = min(best[c], c1[o]);
        } else if (staged) {
#pragma unroll
            for (int k = 0; k < NST; ++k) {
                const int32_t q = (int32_t)threadIdx.x + FT * k;
                if (q < H + FC) {
                    seg[q] = mbase - H + q >= -padl ? stv[k] : DINF;
                    if (sweep) seg3[q] = stv3[k];
                }
            }
            __syncthreads();
            const int32_t *const sg = seg + H + (ml - mbase);  // column ml
            if (m0 >= ch.need1max[s]) {
                for (int32_t o = 0; o < K; ++o) {
                    const int32_t *const so = sg - xbar[o];
#pragma unroll
                    for (int c = 0; c < NC; ++c) best[c] = min(best[c], c1[o] + so[64 * c]);
                }
            } else {
                for (int32_t o = 0; o < K; ++o) {
                    const int32_t *const so = sg - xbar[o];
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        if (ml + 64 * c >= need1[o]) best[c] = min(best[c], c1[o] + so[64 * c]);
                }
            }
            if (sweep) {
                const int32_t *const sg3 = seg3 + H + (ml - mbase);
                for (int32_t o = 0; o < K; ++o) {
                    const int32_t *const so = sg3 - (xbar[o] - x1);
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        if (ml + 64 * c >= need1[o]) best[c] = min(best[c], c3[o] + so[64 * c]);
                }
            }
        } else {
            for (int32_t o = 0; o < K; ++o)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    if (ml + 64 * c >= need1[o]) best[c] = min(best[c], c1[o] + ldb(rest - xbar[o], col[c]));
            if (sweep)
                for (int32_t o = 0; o < K; ++o)
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        if (ml + 64 * c >= need1[o])
                            best[c] = min(best[c], c3[o] + ldb(hrest - (xbar[o] - x1), col[c]));
        }
        if (run2)  // the second near range, loaded before case 1
#pragma unroll
            for (int u = 0; u < FB; ++u)
#pragma unroll
                for (int c = 0; c < NC; ++c) best[c] = min(best[c], va2[u][c] + vq2[u][c]);
    } else if (chunk >= n_run_h) {
        // past msaH(s,t) of every cell of the diagonal: H(s,t) = lb(s,t) + P[s][s+1] (the
        // lower bound of every candidate, reached by split s+1); the products did not run here
        const int32_t hv = ch.lb[row_st] + ch.P[(int64_t)s * L + s + 1];
#pragma unroll
        for (int c = 0; c < NC; ++c) best[c] = hv;
    } else {
        // H(s, t) = min_i aq(s, i, m - x_s) + Opt(i, t, m - x_i): the products' partial, then
        // the near splits
        const int32_t *const hrow = tb.hopt + row_st * stride + padl;
#pragma unroll
        for (int c = 0; c < NC; ++c) best[c] = D > 0 ? ldb(hrow, col[c]) : DINF;
        near_first(tb.aq, min(ch.x[s], padl));
        near_second(tb.aq, min(ch.x[s], padl));
    }

    // stores last: until here every scalar operand may come from the scalar cache
    if (hp) {
        int32_t *const hrow = tb.hopt + row_st * stride + padl;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int32_t m = ml + 64 * c;
            if (m < W) st_nt(min(best[c], DINF), &hrow[m]);
        }
        return;
    }
    // Opt, its copy in the right operand table (Opt(s, t, m) at column m + x_s, infinity
    // below x_s), the left operand ap(s, t+1) of Eq. fn and, with the saving sweep, the left
    // operand aq(s, t+1, v) = P[s][t+1] + Opt(s, t, v) of H(s, .) if the sweep s..t fits v + x_s
    int32_t *const srow = p_os + row_st * stride + padl;
    int32_t *const arow = p_ap + row_st * stride + padl;
    int32_t *const qrow = tb.aq ? tb.aq + row_st * stride + padl : nullptr;
    const int32_t need2 = t + 1 < L ? ch.need2[ip] : 0, P = t + 1 < L ? ch.P[ip] : 0;
    const int32_t need3 = qrow && t + 1 < L ? ch.need3[ip] : 0, xs = ch.x[s];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int32_t m = ml + 64 * c;
        if (m < padl) {  // keep the left pads infinite
            st_nt(DINF, &orow[m - padl]);
            if (qrow) st_nt(DINF, &qrow[m - padl]);
        }
        if (m < W) {
            const int32_t v = min(best[c], DINF);
            st_nt(v, &orow[m]);
            if (m < xs) st_nt(DINF, &srow[m]);
            if ((int64_t)m + xs < W) st_nt(v, &srow[m + xs]);
            if (t + 1 < L) {
                st_nt(m >= need2 ? min(P + v, DINF) : DINF, &arow[m]);
                if (qrow) st_nt(m + xs >= need3 ? min(P + v, DINF) : DINF, &qrow[m]);
            }
        }
    }
}

// Relaxations (real split candidates) one product launch covers: cells of spans dd in
// [tau, tau + T) whose split has a left span a and a right span dd-1-a in the given windows.
static int64_t product_work(int32_t L, int32_t W, int32_t tau, int32_t T, int32_t alo, int32_t ahi,
                            int32_t blo, int32_t bhi)
{
    int64_t n = 0;
    for (int32_t dd = tau; dd < min(tau + T, L); ++dd) {
        int64_t c = 0;
        for (int32_t a = alo; a < min(ahi, dd); ++a) c += (dd - 1 - a >= blo && dd - 1 - a < bhi);
        n += (int64_t)(L - dd) * c;
    }
    return n * W;
}

// What a product launch does, column chunk by column chunk: cap(s, t, mc) = 0 when the tile
// of cell (s, t) does not run on 64-column chunk mc, else the first split past those the
// cell relaxes there (INT32_MAX: all of them).  Adds the relaxations evaluated and the
// compulsory table traffic of what runs: per chunk, the distinct ap rows (s, s+a) and Opt
// rows (t-b, t) some relaxed candidate reads, plus the target rows written (and read back
// when folding into a stored partial).  Chunks whose cells run exactly as on the previous
// chunk repeat its counts.
template <class F>
static void tile_account(int32_t L, int32_t W, int32_t tau, int32_t T, int32_t alo, int32_t ahi, int32_t blo,
                         int32_t bhi, bool accumulate, int32_t n_run, F cap, int64_t *work, int64_t *bytes)
{
    const int32_t dmax = min(tau + T, L);
    std::vector<int32_t> caps, prev;
    std::vector<std::pair<int32_t, int32_t>> iv;
    int64_t c_work = 0, c_rows = 0;  // per column of the previous chunk
    for (int32_t mc = 0; mc < n_run && 64 * mc < W; ++mc) {
        caps.clear();
        for (int32_t s = 0; s < L - tau; ++s)
            for (int32_t dd = tau; dd < min(dmax, L - s); ++dd) caps.push_back(cap(s, s + dd, mc));
        const int64_t cols = min(64, W - 64 * mc);
        if (mc == 0 || caps != prev) {
            c_work = c_rows = 0;
            // split a of cell (s, s+dd) is real for a in [alo, ahi), b = dd-1-a in [blo, bhi), and
            // relaxed for i = s+1+a < cap
            auto arange = [&](int32_t s, int32_t dd, int32_t c, int32_t *a0, int32_t *a1) {
                *a0 = max(alo, dd - bhi);
                *a1 = min(min(ahi - 1, dd - 1 - blo), c == INT32_MAX ? INT32_MAX : c - 2 - s);
            };
            size_t q = 0;
            for (int32_t s = 0; s < L - tau; ++s) {  // ap rows: the a intervals grow with dd
                int32_t lo = 0, hi = -1;
                for (int32_t dd = tau; dd < min(dmax, L - s); ++dd) {
                    const int32_t c = caps[q++];
                    if (c == 0) continue;
                    c_rows += accumulate ? 2 : 1;  // the target row written (and read back)
                    int32_t a0, a1;
                    arange(s, dd, c, &a0, &a1);
                    if (a0 > a1) continue;
                    c_work += a1 - a0 + 1;
                    if (hi < lo) lo = a0, hi = a1;
                    else if (a0 <= hi + 1) hi = max(hi, a1);
                    else c_rows += hi - lo + 1, lo = a0, hi = a1;
                }
                if (hi >= lo) c_rows += hi - lo + 1;
            }
            for (int32_t t = tau; t < L; ++t) {  // Opt rows: intervals of b, merged after sorting
                iv.clear();
                for (int32_t dd = tau; dd < min(dmax, t + 1); ++dd) {
                    const int32_t s = t - dd;
                    const int32_t c = cap(s, t, mc);
                    if (c == 0) continue;
                    int32_t a0, a1;
                    arange(s, dd, c, &a0, &a1);
                    if (a0 <= a1) iv.emplace_back(dd - 1 - a1, dd - 1 - a0);
                }
                std::sort(iv.begin(), iv.end());
                int32_t lo = 0, hi = -1;
                for (const auto &v : iv) {
                    if (hi < lo) lo = v.first, hi = v.second;
                    else if (v.first <= hi + 1) hi = max(hi, v.second);
                    else c_rows += hi - lo + 1, lo = v.first, hi = v.second;
                }
                if (hi >= lo) c_rows += hi - lo + 1;
            }
            prev.swap(caps);
        }
        *work += c_work * cols;
        *bytes += c_rows * cols * 4;
    }
}

// 64-column chunks a product or mid launch runs when its target cells' largest msa is sat:
// whole finalize workgroups (FC = 128 columns), so that every column a finalize computes
// from operands has its partial.
static inline int32_t run_chunks(int32_t sat) { return (int32_t)(((int64_t)sat + 127) / 128 * 2); }

template <int WD>
static hipError_t launch_mid(const DevChain &ch, const Tables &tb, hipStream_t stream, int32_t d,
                             int32_t *n, Profiler *prof)
{
    hipError_t e;
    const int32_t lo = d - WD, L = ch.L;
    constexpr int R = mid_rows<WD>();
    const int32_t n_blk = (L - d + R - 1) / R, n_mc = (tb.W + 63) / 64;
    // column chunks below the largest msa of the target spans [d, d + WD) (msa grows with t)
    int32_t sat = 0;
    for (int32_t s = 0; s < L - d; ++s) sat = max(sat, ch.h_msa[row_of(L, s, min(s + d + WD - 1, L - 1))]);
    const int32_t n_chunks = min(n_mc, run_chunks(sat));
    int32_t n_chunks_h = 0;  // H of the saving sweep: the chunks below the largest msaH
    if (tb.hopt) {
        int32_t sat_h = 0;
        for (int32_t s = 0; s < L - d; ++s) sat_h = max(sat_h, ch.h_msaH[row_of(L, s, min(s + d + WD - 1, L - 1))]);
        n_chunks_h = min(n_mc, run_chunks(sat_h));
    }
    const int64_t w1 = lo == 0 ? product_work(L, tb.W, d, WD, 0, WD, 0, WD)
                               : product_work(L, tb.W, d, WD, lo, d, 0, d) + product_work(L, tb.W, d, WD, 0, lo, lo, d);
    prof->work[KFILL_MID] += w1 * (tb.hopt ? 2 : 1);
    if (n_chunks + n_chunks_h == 0) return hipSuccess;  // every target cell is past msa: the finalize stores it
    const int32_t n_groups = lo == 0 ? 1 : 2;
    const dim3 grid(chunk_grid(n_chunks + n_chunks_h, n_groups * n_blk));
    const bool cnt = tb.ctr != nullptr;
    const int64_t n_rec = (int64_t)(n_chunks + n_chunks_h) * n_groups * n_blk;
    Tables tr = tb;
    if (cnt) {
        if ((e = prof->records(stream, n_rec)) != hipSuccess) return e;
        tr.rec = prof->d_rec;
    }
    const uint32_t tpack = (uint32_t)d | (uint32_t)(lo > 0) << 11;  // d < 2048
    e = lo == 0 ? launch(prof, KFILL_MID, cnt ? k_mid<WD, true, true> : k_mid<WD, true, false>, grid, dim3(64),
                         stream, tr.opt, tr.os, tr.ap, (int32_t)tr.stride, tr.padl, tr.W, ch.L, (int32_t)tr.inf_row,
                         tpack, n_chunks + n_chunks_h, n_chunks, ch, tr, n_chunks_h)
                : launch(prof, KFILL_MID, cnt ? k_mid<WD, false, true> : k_mid<WD, false, false>, grid, dim3(64),
                         stream, tr.opt, tr.os, tr.ap, (int32_t)tr.stride, tr.padl, tr.W, ch.L, (int32_t)tr.inf_row,
                         tpack, n_chunks + n_chunks_h, n_chunks, ch, tr, n_chunks_h);
    if (e != hipSuccess) return e;
    ++*n;
    if (prof->on) {
        // what runs: every tile on the launch's first n_chunks column chunks (H: all); with the
        // records, only the tiles that ran.  A group A tile holds the cells of R rows, a group
        // B tile those of R ends.
        if (cnt && (e = prof->read_records(stream, n_rec)) != hipSuccess) return e;
        for (int32_t part = 0; part < 2; ++part) {  // Opt's chunks, then H's
            const int32_t k = part ? n_chunks_h : n_chunks, c0 = part ? n_chunks : 0;
            if (k == 0) continue;
            auto cap = [&](int32_t grp) {
                return [&, grp](int32_t s, int32_t t, int32_t mc) -> int32_t {
                    if (mc >= k) return 0;
                    if (!cnt) return INT32_MAX;
                    const int32_t blk = grp == 0 ? s / R : (t - d) / R;
                    return prof->h_rec[((int64_t)(c0 + mc) * n_groups + grp) * n_blk + blk] ? INT32_MAX : 0;
                };
            };
            int64_t *w = &prof->eval[KFILL_MID], *by = &prof->bytes[KFILL_MID];
            if (lo == 0) {
                tile_account(L, tb.W, d, WD, 0, WD, 0, WD, false, k, cap(0), w, by);
            } else {
                tile_account(L, tb.W, d, WD, lo, d, 0, d, true, k, cap(0), w, by);
                tile_account(L, tb.W, d, WD, 0, lo, lo, d, true, k, cap(1), w, by);
            }
        }
    }
    return hipSuccess;
}

// The fill: per diagonal d, the products that complete before it (a band product every
// BAND spans, mid products in between down to width midmin), then its finalize.
hipError_t launch_fill(const DevChain &ch, const Tables &tb, hipStream_t stream, int32_t *launches,
                       Profiler *prof)
{
    static_assert(BAND == 32, "the launch sequence below is written for 32-span bands");
    hipError_t e;
    int32_t n = 0;
    const int32_t midmin = MIDMIN;
    e = launch(prof, KFILL_INIT, k_init_inf_rows, dim3((tb.stride + 255) / 256, (tb.hopt ? 5 : 3) * (2 * SLACK + 1)),
               dim3(256), stream, tb);
    if (e != hipSuccess) return e;
    ++n;
    const int32_t fin_x = (max(tb.W, tb.padl) + FC - 1) / FC;
    for (int32_t d = 0; d < ch.L; ++d) {
        if (d > 0 && d % BAND == 0) {
            constexpr int SR = 4, TW = 16, TH = 2, NW = 4, SW = SR * NW / TH;  // product tile
            int32_t sat = 0;  // column chunks below the largest msa of the band's spans
            for (int32_t s = 0; s < ch.L - d; ++s)
                sat = max(sat, ch.h_msa[row_of(ch.L, s, min(s + d + BAND - 1, ch.L - 1))]);
            const int32_t n_chunks = min((tb.W + 63) / 64, run_chunks(sat));
            int32_t n_chunks_h = 0;  // H of the saving sweep: the chunks below the largest msaH
            if (tb.hopt) {
                int32_t sat_h = 0;
                for (int32_t s = 0; s < ch.L - d; ++s)
                    sat_h = max(sat_h, ch.h_msaH[row_of(ch.L, s, min(s + d + BAND - 1, ch.L - 1))]);
                n_chunks_h = min((tb.W + 63) / 64, run_chunks(sat_h));
            }
            prof->work[KFILL_PRODUCT] += product_work(ch.L, tb.W, d, BAND, 0, d, 0, d) * (tb.hopt ? 2 : 1);
            const int32_t n_rb = (ch.L - d + SW - 1) / SW;  // row blocks: a workgroup holds SW rows
            const bool cnt = tb.ctr != nullptr;
            const int64_t n_rec = (int64_t)(n_chunks + n_chunks_h) * n_rb;
            if (n_chunks + n_chunks_h > 0) {
                const dim3 grid(chunk_grid(n_chunks + n_chunks_h, n_rb));
                auto *const kp = cnt ? k_product<SR, TW, TH, NW, true> : k_product<SR, TW, TH, NW, false>;
                Tables tr = tb;
                if (cnt) {
                    if ((e = prof->records(stream, n_rec)) != hipSuccess) return e;
                    tr.rec = prof->d_rec;
                }
                e = launch(prof, KFILL_PRODUCT, kp, grid, dim3(NW * 64), stream, ch, tr, d, n_chunks, n_chunks_h);
                if (e != hipSuccess) return e;
                ++n;
                if (cnt && (e = prof->read_records(stream, n_rec)) != hipSuccess) return e;
            }
            if (prof->on) {
                // every tile on the launch's first n_chunks column chunks (H: all), relaxing all
                // its splits or, with the records, those below the recorded one
                for (int32_t part = 0; part < 2; ++part) {  // Opt's chunks, then H's
                    const int32_t k = part ? n_chunks_h : n_chunks, c0 = part ? n_chunks : 0;
                    if (k == 0) continue;
                    auto cap = [&](int32_t s, int32_t, int32_t mc) -> int32_t {
                        if (mc >= k) return 0;
                        return cnt ? prof->h_rec[(int64_t)(c0 + mc) * n_rb + s / SW] : INT32_MAX;
                    };
                    tile_account(ch.L, tb.W, d, BAND, 0, d, 0, d, false, k, cap, &prof->eval[KFILL_PRODUCT],
                                 &prof->bytes[KFILL_PRODUCT]);
                }
            }
        } else if (d % 16 == 0 && d > 0) {
            if ((e = launch_mid<16>(ch, tb, stream, d, &n, prof)) != hipSuccess) return e;
        } else if (d % 8 == 0 && d > 0) {
            if ((e = launch_mid<8>(ch, tb, stream, d, &n, prof)) != hipSuccess) return e;
        }
        int32_t sat = 0;  // chunks from n_run on lie past every cell's msa: they only store
        for (int32_t s = 0; s + d < ch.L; ++s) sat = max(sat, ch.h_msa[row_of(ch.L, s, s + d)]);
        const int32_t n_run = (int32_t)std::min<int64_t>(fin_x, ((int64_t)sat + FC - 1) / FC);
        const int32_t fin_h = tb.hopt && d >= 1 ? fin_x : 0;  // H(s, s+d) of the saving sweep
        int32_t n_run_h = 0;  // H's chunks from n_run_h on lie past every cell's msaH: they only store
        if (fin_h) {
            int32_t sat_h = 0;
            for (int32_t s = 0; s + d < ch.L; ++s) sat_h = max(sat_h, ch.h_msaH[row_of(ch.L, s, s + d)]);
            n_run_h = (int32_t)std::min<int64_t>(fin_x, ((int64_t)sat_h + FC - 1) / FC);
        }
        const uint32_t dpack = (uint32_t)d | (uint32_t)(d / midmin * midmin) << 11 |
                               (uint32_t)(ch.c3 != nullptr) << 22 | (uint32_t)std::min(ch.xbar_halo, 511) << 23;
        e = launch(prof, KFILL_FINALIZE, tb.ctr ? k_finalize<true> : k_finalize<false>,
                   dim3(chunk_grid(fin_x + fin_h, ch.L - d)), dim3(FT), stream, tb.opt, tb.os, tb.ap, dpack,
                   fin_x + fin_h, fin_x, n_run, ch.L, tb.W, tb.padl, (int32_t)tb.stride, ch, tb, n_run_h);
        if (e != hipSuccess) return e;
        ++n;
        const int32_t D = (d / midmin) * midmin, near = D > 0 ? 2 * (d - D) : d;
        // per cell: Opt's near splits and options; with the sweep also H's near splits and
        // case 3's options
        const int64_t per_cell = near + ch.K + (tb.hopt ? near + (d >= 2 ? ch.K : 0) : 0);
        prof->work[KFILL_FINALIZE] += (int64_t)(ch.L - d) * per_cell * tb.W;
        if (prof->on) {
            // per cell, in the workgroups below msa: two operand rows per split, the stored
            // partial, the case-1 row, the Opt row written; past msa only the Opt row
            // written; and everywhere the right operand row written, and the ap row (with the
            // saving sweep also the aq row) where a later split uses it.  With the saving
            // sweep, H's workgroups (every column, d >= 1): two operand rows per split, the
            // stored partial and the H row written.
            for (int32_t s = 0; s + d < ch.L; ++s) {
                const int64_t run = std::min<int64_t>(tb.W, (int64_t)n_run * FC);
                const int64_t run_h = std::min<int64_t>(tb.W, (int64_t)n_run_h * FC);
                prof->eval[KFILL_FINALIZE] += run * (near + ch.K + (tb.hopt && d >= 2 ? ch.K : 0)) + run_h * near;
                prof->bytes[KFILL_FINALIZE] +=
                    (run * (2 * near + (D > 0) + (d > 0) + 1) + (tb.W - run) + tb.W +
                     (s + d + 1 < ch.L ? (int64_t)tb.W * (tb.aq ? 2 : 1) : 0) +
                     (fin_h ? run_h * (2 * near + (D > 0)) + tb.W : 0)) * 4;
            }
        }
    }
    *launches = n;
    return hipSuccess;
}

// ---------------------------------------------------------------------------------------
// Choice recovery.  The key of a candidate is (cost << 32) | code, so the smallest key is
// the lexicographic (cost, code) minimum; invalid or infinite candidates get ~0.
// ---------------------------------------------------------------------------------------
__device__ inline int32_t opt_at(const Tables &tb, int32_t L, int32_t s, int32_t t, int32_t m)
{
    return tb.opt[row_of(L, s, t) * tb.stride + tb.padl + m];
}

__device__ inline uint64_t split_key(const DevChain &ch, const Tables &tb, int32_t s, int32_t t,
                                     int32_t m, int32_t i)
{
    const int32_t L = ch.L;
    if (m < ch.need2[s * L + i]) return ~0ull;
    const int32_t a = opt_at(tb, L, s, i - 1, m);
    const int32_t q = opt_at(tb, L, i, t, m - ch.x[i]);
    if (a >= DINF || q >= DINF) return ~0ull;
    const int64_t v = (int64_t)ch.P[s * L + i] + a + q;
    if (v >= DINF) return ~0ull;
    return ((uint64_t)v << 32) | (uint32_t)i;
}

__device__ inline uint64_t option_key(const DevChain &ch, const Tables &tb, int32_t s, int32_t t,
                                      int32_t m, int32_t o)
{
    const int32_t L = ch.L, K = ch.K;
    if (m < ch.need1[s * K + o]) return ~0ull;
    int32_t rest = 0;
    if (t > s) rest = opt_at(tb, L, s + 1, t, m - ch.xbar[s * K + o]);
    if (rest >= DINF) return ~0ull;
    const int64_t v = (int64_t)ch.c1[s * K + o] + rest;
    if (v >= DINF) return ~0ull;
    return ((uint64_t)v << 32) | (uint32_t)(L + o);
}

// Case 3 (the saving sweep) with option slot o: code L + K + o.
__device__ inline uint64_t sweep_key(const DevChain &ch, const Tables &tb, int32_t s, int32_t t,
                                     int32_t m, int32_t o)
{
    const int32_t L = ch.L, K = ch.K;
    if (!ch.c3 || t < s + 2 || m < ch.need1[s * K + o]) return ~0ull;
    const int32_t mem = ch.xbar[s * K + o] - ch.x[s + 1];
    const int32_t h = tb.hopt[row_of(L, s + 1, t) * tb.stride + tb.padl + (m - mem)];
    if (h >= DINF) return ~0ull;
    const int64_t v = (int64_t)ch.c3[s * K + o] + h;
    if (v >= DINF) return ~0ull;
    return ((uint64_t)v << 32) | (uint32_t)(L + K + o);
}

// One row of choice codes: thread m scans the candidates in code order.
__global__ __launch_bounds__(256) void k_arg_row(DevChain ch, Tables tb, int32_t s, int32_t t,
                                                 int16_t *__restrict__ out)
{
    const int32_t m = blockIdx.x * 256 + threadIdx.x;
    if (m >= tb.W) return;
    uint64_t best = ~0ull;
    for (int32_t i = s + 1; i <= t; ++i) best = min(best, split_key(ch, tb, s, t, m, i));
    for (int32_t o = 0; o < ch.K; ++o) best = min(best, option_key(ch, tb, s, t, m, o));
    if (ch.c3)
        for (int32_t o = 0; o < ch.K; ++o) best = min(best, sweep_key(ch, tb, s, t, m, o));
    out[m] = best == ~0ull ? (int16_t)-1 : (int16_t)(best & 0xffffu);
}

hipError_t launch_arg_row(const DevChain &ch, const Tables &tb, int32_t s, int32_t t, int16_t *out,
                          hipStream_t stream)
{
    hipLaunchKernelGGL(k_arg_row, dim3((tb.W + 255) / 256), dim3(256), 0, stream, ch, tb, s, t, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Alg. 3 (rk-Rotor-Build) with an explicit stack, one wavefront.  Every lane keeps the
// same stack copy in LDS (all lanes write identical frames), so no barrier is needed;
// the lanes share only the choice search at each visited cell.
// ---------------------------------------------------------------------------------------
struct Frame { int32_t type, a, b, c; };  // type 0: Build(s=a, t=b, m=c); 1: emit (kind=a, block=b, option=c)
static_assert(sizeof(Frame) == 4 * sizeof(int32_t), "frames are four int32 in LDS");

// Minimum of a 32-bit value over the 64 lanes of a wavefront (all lanes active): DPP
// exchanges inside each row of 16 lanes (swap neighbours, swap pairs, rotate by 4 and by 8)
// leave the row's minimum in every lane; the four row minima are then read as scalars.
__device__ inline uint32_t wave_min_u32(uint32_t v)
{
    v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xb1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
    v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4e, 0xf, 0xf, false));   // quad_perm 2,3,0,1
    v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x124, 0xf, 0xf, false));  // row_ror 4
    v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xf, 0xf, false));  // row_ror 8
    const uint32_t r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return min(min(r0, r1), min(r2, r3));
}

// Per visited cell, the lanes evaluate its candidates in parallel with one round of
// independent loads: a split's left operand comes from ap (which already holds P, the
// sweep's validity and the saturation), its right operand from Opt at the shifted column;
// an option's rest from Opt.  The activation sizes (and the options' xbar, when it fits)
// are copied to LDS first, so no load waits on another.  Shifted columns are clamped into
// the row's left pad: a candidate whose column would fall left of it is invalid.
constexpr int32_t BT_XBAR_LDS_MAX = 8192;  // xbar entries kept in LDS (32 KiB)
// Frames on the stack: every step pushes at most 2 per block its span loses (case 3 pushes
// 4 and loses at least 2 blocks).
__host__ __device__ inline int32_t bt_stack_cap(const DevChain &ch) { return (ch.c3 ? 4 : 2) * ch.L + 8; }

template <bool XBAR_LDS>
__global__ __launch_bounds__(64) void k_backtrace(DevChain ch, Tables tb, int32_t m_top,
                                                  rk_op *__restrict__ ops, int64_t cap,
                                                  int64_t *__restrict__ res)
{
    extern __shared__ int32_t sh[];
    const int32_t lane = threadIdx.x, L = ch.L, K = ch.K;
    const int32_t stack_cap = bt_stack_cap(ch);
    const bool sweep = ch.c3 != nullptr;
    Frame *const stk = reinterpret_cast<Frame *>(sh);
    int32_t *const xs = sh + 4 * stack_cap;  // x_0..x_L
    int32_t *const xbs = xs + (L + 1);
    for (int32_t j = lane; j <= L; j += 64) xs[j] = ch.x[j];
    if (XBAR_LDS)
        for (int32_t j = lane; j < L * K; j += 64) xbs[j] = ch.xbar[j];
    __syncthreads();
    const int32_t *const xbar = XBAR_LDS ? xbs : ch.xbar;
    const int64_t stride = tb.stride;
    const int32_t padl = tb.padl;
    int32_t sp = 0;
    int64_t n = 0, nfwd = -1, status = 0;

    auto emit = [&](int32_t kind, int32_t block, int32_t option) {
        if (kind == RK_BWD && nfwd < 0) nfwd = n;
        if (lane == 0 && n < cap) ops[n] = rk_op{kind, block, option};
        ++n;
    };
    auto push = [&](Frame f) { stk[sp] = f; ++sp; };

    // The cell being resolved stays in registers; the stack holds what comes after it.
    int32_t s = 0, t = L - 1, m = m_top;
    bool have = true;
    for (;;) {
        if (!have) {
            if (sp == 0) break;
            const Frame f = stk[--sp];
            if (f.type == 1) { emit(f.a, f.b, f.c); continue; }
            s = f.a; t = f.b; m = f.c;
        }
        const int32_t d = t - s;
        const int32_t own = tb.opt[row_of(L, s, t) * stride + padl + m];
        // This lane's smallest (cost, code) key over its candidates: split i = s+1+j (j < d)
        // has code i, option o has code L+o.  Addresses of candidates past the end are
        // clamped into the tables; their values are then ignored.  Row numbers fit 32 bits
        // (L <= 2000), so each address is one 32x32+64 multiply-add from the table base.
        uint64_t best = ~0ull;
        auto take = [&](bool ok, uint32_t v, uint32_t code) {
            const uint64_t key = ok ? ((uint64_t)v << 32) | code : ~0ull;
            best = key < best ? key : best;
        };
        auto row32 = [&](int32_t a, int32_t b) { return (uint32_t)(a * L - ((a * (a - 1)) >> 1) + b - a); };
        const uint32_t ustride = (uint32_t)stride;
        const int32_t *const ap_s = tb.ap + (uint64_t)row32(s, s) * ustride + padl + m;
        const int32_t rest_row = row32(min(s + 1, t), t);
        // NB split candidates per lane and round of loads: as many as the cell has splits
        // (up to 8 per lane), so short spans do not pay for the longest ones
        auto cell = [&](auto nbc) {
        constexpr int NB = decltype(nbc)::value;
        const int32_t rounds = max((d + 64 * NB - 1) / (64 * NB), (K + 63) / 64);
        for (int32_t r = 0; r < rounds; ++r) {
            // the option's xbar first: when it comes from global memory, the rest's address
            // waits for it alone, not for the splits' loads
            const int32_t o = r * 64 + lane, ko = s * K + min(o, K - 1);
            const int32_t xb = xbar[ko];
            int32_t xi[NB], av[NB], qv[NB];
#pragma unroll
            for (int u = 0; u < NB; ++u) xi[u] = xs[min(s + 1 + r * 64 * NB + 64 * u + lane, t)];
#pragma unroll
            for (int u = 0; u < NB; ++u) {
                const int32_t jc = min(r * 64 * NB + 64 * u + lane, max(d - 1, 0));
                const int32_t i = min(s + 1 + jc, t);
                av[u] = ap_s[(uint64_t)(uint32_t)jc * ustride];
                qv[u] = tb.opt[(uint64_t)row32(i, t) * ustride + (uint32_t)(padl + m - min(xi[u], padl))];
            }
            const int32_t c1 = ch.c1[ko], need = ch.need1[ko];
            const int32_t rest_v = tb.opt[(uint64_t)rest_row * ustride + (uint32_t)(padl + max(m - xb, -padl))];
            const int32_t rest = t > s ? rest_v : 0;  // row (s, s) stands in when t == s
#pragma unroll
            for (int u = 0; u < NB; ++u) {
                const int32_t j = r * 64 * NB + 64 * u + lane;
                take(j < d, (uint32_t)av[u] + (uint32_t)qv[u], (uint32_t)(s + 1 + j));
            }
            take(o < K && m >= need, (uint32_t)c1 + (uint32_t)rest, (uint32_t)(L + o));
            if (sweep) {  // case 3 with option o: c3 + H(s+1, t, m - mem), mem = xbar - x_{s+1}
                const int32_t hv =
                    tb.hopt[(uint64_t)rest_row * ustride + (uint32_t)(padl + max(m - (xb - xs[s + 1]), 0))];
                take(o < K && m >= need && t >= s + 2, (uint32_t)ch.c3[ko] + (uint32_t)hv, (uint32_t)(L + K + o));
            }
        }
        };
        if (d <= 64) cell(std::integral_constant<int, 1>{});
        else if (d <= 128) cell(std::integral_constant<int, 2>{});
        else if (d <= 256) cell(std::integral_constant<int, 4>{});
        else cell(std::integral_constant<int, 8>{});
        const uint32_t bc = (uint32_t)(best >> 32), bk = (uint32_t)best;
        const uint32_t cost = wave_min_u32(bc);
        const uint32_t code = wave_min_u32(bc == cost ? bk : ~0u);
        if (cost >= (uint32_t)DINF) { status = 1; break; }
        if ((int32_t)cost != own) { status = 2; break; }
        if (sp + 4 > stack_cap) { status = 3; break; }
        if (code >= (uint32_t)(L + K)) {
            // case 3: F_s^o keeps its data; the sweep s+1..i-1 to x_i, where i is H's choice at
            // (s+1, t, u = m - mem); then i..t, x_i dropped, x_{s+1} made again from the kept
            // data, s+1..i-1, and B_s^o
            const int32_t o = (int32_t)code - L - K, s1 = s + 1;
            const int32_t xb = xbar[s * K + o];
            const int32_t u = m - (xb - xs[s1]);
            const int32_t hown = tb.hopt[row_of(L, s1, t) * stride + padl + u];
            const int32_t *const aq_s = tb.aq + (uint64_t)row32(s1, s1) * ustride + padl + u - min(xs[s1], padl);
            uint64_t hb = ~0ull;
            for (int32_t j = lane; j < t - s1; j += 64) {  // split i = s1 + 1 + j, code i
                const int32_t i = s1 + 1 + j;
                const int32_t a = aq_s[(uint64_t)(uint32_t)j * ustride];
                const int32_t q = tb.opt[(uint64_t)row32(i, t) * ustride + (uint32_t)(padl + u - min(xs[i], padl))];
                hb = min(hb, ((uint64_t)((uint32_t)a + (uint32_t)q) << 32) | (uint32_t)i);
            }
            const uint32_t hc = (uint32_t)(hb >> 32), hk = (uint32_t)hb;
            const uint32_t hcost = wave_min_u32(hc);
            const int32_t i = (int32_t)wave_min_u32(hc == hcost ? hk : ~0u);
            if ((int32_t)hcost != hown || hcost >= (uint32_t)DINF || i <= s1 || i > t) { status = 2; break; }
            emit(RK_FWD_SAVE, s, o);
            for (int32_t k = lane; k < i - s - 1; k += 64) {
                const int64_t at = n + 2 * (int64_t)k;
                if (at < cap) ops[at] = rk_op{RK_FWD_NOSAVE, s1 + k, -1};
                if (at + 1 < cap) ops[at + 1] = rk_op{RK_FREE_X, s1 + k, -1};
            }
            n += 2 * (int64_t)(i - s - 1);
            push(Frame{1, RK_BWD, s, o});
            push(Frame{0, s1, i - 1, m - xb});
            push(Frame{1, RK_REFWD, s, o});
            push(Frame{1, RK_FREE_X, i, -1});
            have = true;
            s = i;
            m = u - xs[i];
        } else if (code >= (uint32_t)L) {
            const int32_t o = (int32_t)code - L;
            emit(RK_FWD_SAVE, s, o);
            push(Frame{1, RK_BWD, s, o});
            have = t > s;
            m -= xbar[s * K + o];
            s += 1;
        } else {
            // forward through blocks s..i-1 keeping nothing, dropping x_{s+1}..x_{i-1} behind
            const int32_t i = (int32_t)code;
            emit(RK_FWD_NOSAVE, s, -1);
            for (int32_t k = lane; k < i - s - 1; k += 64) {
                const int64_t at = n + 2 * (int64_t)k;
                if (at < cap) ops[at] = rk_op{RK_FWD_NOSAVE, s + 1 + k, -1};
                if (at + 1 < cap) ops[at + 1] = rk_op{RK_FREE_X, s + 1 + k, -1};
            }
            n += 2 * (int64_t)(i - s - 1);
            push(Frame{0, s, i - 1, m});
            push(Frame{1, RK_FREE_X, i, -1});
            have = true;
            s = i;
            m -= xs[i];
        }
    }
    if (lane == 0) {
        res[0] = n;
        res[1] = nfwd;
        res[2] = status;
    }
}

hipError_t launch_backtrace(const DevChain &ch, const Tables &tb, int32_t m_top, rk_op *ops,
                            int64_t cap, int64_t *res, hipStream_t stream)
{
    const bool xbar_lds = (int64_t)ch.L * ch.K <= BT_XBAR_LDS_MAX;
    const size_t lds = sizeof(Frame) * (size_t)bt_stack_cap(ch) + sizeof(int32_t) * (size_t)(ch.L + 1) +
                       (xbar_lds ? sizeof(int32_t) * (size_t)ch.L * ch.K : 0);
    if (xbar_lds)
        hipLaunchKernelGGL(k_backtrace<true>, dim3(1), dim3(64), lds, stream, ch, tb, m_top, ops, cap, res);
    else
        hipLaunchKernelGGL(k_backtrace<false>, dim3(1), dim3(64), lds, stream, ch, tb, m_top, ops, cap, res);
    return hipGetLastError();
}

}  // namespace rk
