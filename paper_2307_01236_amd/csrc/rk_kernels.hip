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
// Only Opt is stored.  Which choice realises a minimum is recomputed from the
// finished table where it is needed (Alg. 3 does the same: it asks which case
// attains Opt(s,t,m)), so the fill keeps no argmin bookkeeping.
#include "rk_internal.h"

namespace rk {

const char *const kFillKernelNames[KFILL_NKINDS] = {"k_product", "k_finalize", "k_init_inf_rows"};

hipError_t Profiler::before(int32_t kind)
{
    if (!on) return hipSuccess;
    while ((int32_t)events.size() < 2 * (n + 1)) {
        hipEvent_t e;
        hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) return err;
        events.push_back(e);
    }
    kinds.push_back(kind);
    return hipEventRecord(events[2 * n], stream);
}

hipError_t Profiler::after()
{
    if (!on) return hipSuccess;
    hipError_t err = hipEventRecord(events[2 * n + 1], stream);
    ++n;
    return err;
}

// ---------------------------------------------------------------------------------------
// The all-infinity row of both tables (read in place of operands that do not exist yet).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_init_inf_rows(Tables tb)
{
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j < tb.stride) {
        tb.opt[tb.inf_row * tb.stride + j] = DINF;
        tb.ap[tb.inf_row * tb.stride + j] = DINF;
    }
}

// ---------------------------------------------------------------------------------------
// Raw buffer loads: a descriptor per operand block, a fixed per-lane byte offset per row.
// Reads past the descriptor's range return 0 instead of faulting; every such read is
// also one whose value the kernel replaces by infinity.
// ---------------------------------------------------------------------------------------
__device__ inline __amdgpu_buffer_rsrc_t block_rsrc(const int32_t *base, const int32_t *end)
{
    const int64_t bytes = (const char *)end - (const char *)base;
    const uint32_t n = bytes > 0xffffffffll ? 0xffffffffu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)n, 0x00020000);
}

__device__ inline int32_t block_load(__amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, 0);
}

// ---------------------------------------------------------------------------------------
// Workgroups of a launch go to the 8 XCDs round-robin (id g to XCD g mod 8), and each XCD
// has its own L2.  Renumbering them so that every XCD gets one contiguous range of logical
// tiles puts tiles that share operand rows into the same L2 at about the same time.
// A bijection of [0, G); correctness does not depend on the dispatch order.
// ---------------------------------------------------------------------------------------
__device__ inline uint32_t xcd_tile(uint32_t g, uint32_t G)
{
    constexpr uint32_t NX = 8;
    const uint32_t x = g % NX, j = g / NX, base = G / NX, rem = G % NX;
    return (x < rem ? x * (base + 1) : rem * (base + 1) + (x - rem) * base) + j;
}

// ---------------------------------------------------------------------------------------
// Band product.  For the spans d in [tau, tau + T) (one band), the part of Eq. fn over
// the splits i whose two operands are older than the band (both s..i-1 and i..t shorter
// than tau).  That is a min-plus product, elementwise in m:
//     acc(s,t) = min_i ap(s,i) + Opt(i, t, m - x_i).
// A workgroup owns 64 consecutive budgets (lane = m) and SW = 16 consecutive rows s; its
// wave w keeps, per lane, the SR x T accumulators of rows s0..s0+SR-1 (s0 = S0 + SR w)
// and ends t = s + tau + k.  Splits are taken CI at a time.  The right operands
// Opt(i, t, .) of a chunk, for all NQ ends of the workgroup, are staged in LDS (each
// global row read once, then used by up to SR waves x rows); each wave reads its own left
// operands ap(s, i).  The next chunk's operands are fetched into registers while the
// current one is relaxed.  Operands that are not final yet or are not spans become
// infinity; chunks where all operands are known valid skip those checks.
// ---------------------------------------------------------------------------------------
template <int T>
__global__ __launch_bounds__(256) void k_product(DevChain ch, Tables tb, int32_t tau, int32_t x_fit)
{
    constexpr int SR = 4, NW = 4, SW = SR * NW, CI = 4;
    constexpr int NQ = (SW + T - 1 + NW - 1) / NW * NW;  // staged ends, padded to the waves
    constexpr int JW = NQ / NW;                           // staged rows per wave and split
    static_assert(CI % 2 == 0, "splits are relaxed in pairs");
    __shared__ int32_t qs[CI * NQ * 64];

    const int32_t L = ch.L;
    const uint32_t lane = threadIdx.x & 63;
    // wave index as a scalar: every row choice below is wave-uniform
    const int32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t s_end = L - tau;  // rows that own at least one cell of the band
    const uint32_t n_rb = (uint32_t)(s_end + SW - 1) / SW;
    const uint32_t tile = xcd_tile(blockIdx.x, gridDim.x);  // row blocks of a column chunk adjacent
    const int32_t S0 = (int32_t)(tile % n_rb) * SW;
    const uint32_t mchunk = tile / n_rb;
    const int32_t s0 = S0 + wave * SR;
    const int64_t stride = tb.stride;
    const uint32_t m = mchunk * 64 + lane;
    const uint32_t colb = (uint32_t)(tb.padl + min(m, (uint32_t)tb.W - 1)) * 4u;
    const uint32_t pitch = (uint32_t)stride * 4u;
    const int32_t *const opt_end = tb.opt + (tb.inf_row + 1) * stride;
    const int32_t *const ap_end = tb.ap + (tb.inf_row + 1) * stride;
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
            aoff[r] = delta * pitch + colb;
            delta += (uint32_t)(L - 1 - (s0 + r));
        }
    }

    int32_t acc[SR][T];
#pragma unroll
    for (int r = 0; r < SR; ++r)
#pragma unroll
        for (int k = 0; k < T; ++k) acc[r][k] = DINF;

    // fetch(ic) only issues the loads of chunk ic and records, as wave-uniform bit masks,
    // which of them are valid operands; the values are masked when they are first used
    // (one chunk later), so the loads stay in flight while the current chunk is relaxed
    static_assert(CI * JW <= 32 && CI * SR <= 32, "validity masks are 32-bit");
    int32_t qv[CI][JW], av[CI][SR];
    uint32_t qmask = 0, amask = 0;
    auto fetch = [&](int32_t ic) {
        const bool q_core = x_fit && ic + CI - 1 <= i_hi && ic + CI - 1 <= t0 &&
                            t0 + NQ - 1 - ic < tau && t0 + NQ - 1 < L;
        const bool a_core = s0 + SR - 1 < s_end && ic >= s0 + SR && ic + CI - 1 <= s0 + tau &&
                            ic + CI - 1 <= i_hi;
        qmask = 0;
        amask = 0;
#pragma unroll
        for (int ii = 0; ii < CI; ++ii) {
            const int32_t i = ic + ii, ic_ = min(i, L - 1);
            const int32_t xi = ch.x[ic_], xs = min(xi, tb.padl);
            const int32_t *const qb = tb.opt + row_of(L, ic_, t0) * stride - xs;
            const __amdgpu_buffer_rsrc_t rq = block_rsrc(qb, opt_end);
#pragma unroll
            for (int jj = 0; jj < JW; ++jj) {
                qv[ii][jj] = block_load(rq, qoff[jj]);
                const int32_t t = t0 + jj * NW + wave, span = t - i;
                const bool ok = q_core || ((i <= i_hi) & (t < L) & (span >= 0) & (span < tau) &
                                           (xi <= tb.padl));
                qmask |= (uint32_t)ok << (ii * JW + jj);
            }
            const int32_t *const ab = tb.ap + row_of(L, s0, min(i, L) - 1) * stride;
            const __amdgpu_buffer_rsrc_t ra = block_rsrc(ab, ap_end);
#pragma unroll
            for (int r = 0; r < SR; ++r) {
                av[ii][r] = block_load(ra, aoff[r]);
                const int32_t s = s0 + r, span = i - 1 - s;
                const bool ok = a_core || ((i <= i_hi) & (s < s_end) & (span >= 0) & (span < tau));
                amask |= (uint32_t)ok << (ii * SR + r);
            }
        }
    };
    constexpr uint32_t QALL = CI * JW == 32 ? 0xffffffffu : (1u << (CI * JW)) - 1u;
    constexpr uint32_t AALL = CI * SR == 32 ? 0xffffffffu : (1u << (CI * SR)) - 1u;

    const int32_t *const qw = qs + wave * SR * 64 + lane;
    fetch(i_lo);
    for (int32_t ic = i_lo; ic <= i_hi; ic += CI) {
        int32_t a[CI][SR];
        const uint32_t qm = __builtin_amdgcn_readfirstlane(qmask), am = __builtin_amdgcn_readfirstlane(amask);
        if (qm == QALL) {
#pragma unroll
            for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                for (int jj = 0; jj < JW; ++jj) qs[(ii * NQ + jj * NW + wave) * 64 + lane] = qv[ii][jj];
        } else {
#pragma unroll
            for (int ii = 0; ii < CI; ++ii)
#pragma unroll
                for (int jj = 0; jj < JW; ++jj)
                    qs[(ii * NQ + jj * NW + wave) * 64 + lane] =
                        (qm >> (ii * JW + jj)) & 1u ? qv[ii][jj] : DINF;
        }
#pragma unroll
        for (int ii = 0; ii < CI; ++ii)
#pragma unroll
            for (int r = 0; r < SR; ++r)
                a[ii][r] = (am == AALL || ((am >> (ii * SR + r)) & 1u)) ? av[ii][r] : DINF;
        __syncthreads();
        if (ic + CI <= i_hi) fetch(ic + CI);  // in flight while this chunk is relaxed
        // acc(s0+r, s0+r+tau+k) = min(acc, ap(s0+r, i) + Opt(i, s0+r+tau+k, m - x_i)), two splits per min
#pragma unroll
        for (int ii = 0; ii < CI; ii += 2)
#pragma unroll
            for (int r = 0; r < SR; ++r)
#pragma unroll
                for (int k = 0; k < T; ++k)
                    acc[r][k] = min(acc[r][k], min(a[ii][r] + qw[(ii * NQ + r + k) * 64],
                                                   a[ii + 1][r] + qw[((ii + 1) * NQ + r + k) * 64]));
        __syncthreads();
    }
    if (m >= (uint32_t)tb.W) return;
#pragma unroll
    for (int r = 0; r < SR; ++r)
#pragma unroll
        for (int k = 0; k < T; ++k) {
            const int32_t s = s0 + r, t = s + tau + k;
            if (s < s_end && t < L) tb.opt[row_of(L, s, t) * stride + tb.padl + m] = acc[r][k];
        }
}

// ---------------------------------------------------------------------------------------
// Finalize one span-length diagonal d: thread (s, m).  Adds to the band product's
// partial minimum the splits it did not cover (one operand inside the current band:
// max(i-1-s, t-i) >= D, D the band start) and case 1 (Eq. fe), clamps, writes Opt and
// the row's left operand ap(s, t+1) for the spans that will split after t.
// Row pointers advance incrementally (the ap rows of row s are consecutive; the right
// operand row (i+1, t) is L-i-1 rows after (i, t)) and splits go four at a time so their
// loads overlap.  A wave whose smallest budget already satisfies every option's memory
// requirement runs case 1 without per-lane masks.
// ---------------------------------------------------------------------------------------
__device__ inline int32_t row_load(const int32_t *row, uint32_t byte_off)
{
    return *(const int32_t *)((const char *)row + byte_off);
}

__global__ __launch_bounds__(256) void k_finalize(DevChain ch, Tables tb, int32_t d)
{
    const int32_t L = ch.L, K = ch.K;
    const uint32_t n_mc = (uint32_t)(max(tb.W, tb.padl) + 255) / 256;
    const uint32_t tile = xcd_tile(blockIdx.x, gridDim.x);  // column chunks of a row adjacent
    const int32_t s = (int32_t)(tile / n_mc), t = s + d;
    const int32_t mbase = (int32_t)(tile % n_mc) * 256;
    const int32_t m = mbase + (int32_t)threadIdx.x;
    const int32_t m0 = __builtin_amdgcn_readfirstlane(mbase + (int32_t)(threadIdx.x & ~63u));
    const int64_t stride = tb.stride;
    const int32_t padl = tb.padl;
    int32_t *const orow = tb.opt + row_of(L, s, t) * stride;
    if (m < padl) orow[m] = DINF;  // keep the left pad infinite
    if (m >= tb.W) return;
    const uint32_t colb = (uint32_t)(padl + m) * 4u;
    const int32_t D = (d / BAND) * BAND;
    int32_t best = D > 0 ? row_load(orow, colb) : DINF;

    // splits i in [lo, hi]: ap(s, i) + Opt(i, t, m - x_i)
    const int32_t *const aps = tb.ap + row_of(L, s, s) * stride;  // split s+1; split i is i-1-s rows on
    auto splits = [&](int32_t lo, int32_t hi) {
        if (lo > hi) return;
        const int32_t *q = tb.opt + row_of(L, lo, t) * stride;  // row (i, t)
        int32_t i = lo;
        auto one = [&](int32_t ii, const int32_t *qr) {
            const int32_t xi = ch.x[ii];
            const int32_t a = row_load(aps + (int64_t)(ii - 1 - s) * stride, colb);
            const int32_t v = row_load(qr - min(xi, padl), colb);
            return a + (xi <= padl ? v : DINF);
        };
        for (; i + 3 <= hi; i += 4) {
            const int32_t *q1 = q + (int64_t)(L - i - 1) * stride;
            const int32_t *q2 = q1 + (int64_t)(L - i - 2) * stride;
            const int32_t *q3 = q2 + (int64_t)(L - i - 3) * stride;
            const int32_t v0 = one(i, q), v1 = one(i + 1, q1), v2 = one(i + 2, q2), v3 = one(i + 3, q3);
            best = min(best, min(min(v0, v1), min(v2, v3)));
            q = q3 + (int64_t)(L - i - 4) * stride;
        }
        for (; i <= hi; ++i) {
            best = min(best, one(i, q));
            q += (int64_t)(L - i - 1) * stride;
        }
    };
    if (D == 0) {
        splits(s + 1, t);
    } else {
        splits(s + 1, t - D);      // t - i >= D
        splits(s + D + 1, t);      // i - 1 - s >= D
    }

    // case 1, option o: r(F_s^o) + r(B_s^o) + Opt(s+1,t,m-xbar), valid iff m >= need1[s][o]
    const int32_t *const c1 = ch.c1 + s * K, *const need1 = ch.need1 + s * K, *const xbar = ch.xbar + s * K;
    if (d == 0) {
        for (int32_t o = 0; o < K; ++o)
            if (m >= need1[o]) best = min(best, c1[o]);
    } else {
        const int32_t *const rest = tb.opt + row_of(L, s + 1, t) * stride;
        if (m0 >= ch.need1max[s]) {
            int32_t o = 0;
            for (; o + 3 < K; o += 4) {
                const int32_t v0 = c1[o] + row_load(rest - xbar[o], colb);
                const int32_t v1 = c1[o + 1] + row_load(rest - xbar[o + 1], colb);
                const int32_t v2 = c1[o + 2] + row_load(rest - xbar[o + 2], colb);
                const int32_t v3 = c1[o + 3] + row_load(rest - xbar[o + 3], colb);
                best = min(best, min(min(v0, v1), min(v2, v3)));
            }
            for (; o < K; ++o) best = min(best, c1[o] + row_load(rest - xbar[o], colb));
        } else {
            for (int32_t o = 0; o < K; ++o)
                if (m >= need1[o]) best = min(best, c1[o] + row_load(rest - xbar[o], colb));
        }
    }
    best = min(best, DINF);
    orow[padl + m] = best;
    if (t + 1 < L) {
        const int32_t i = t + 1;
        tb.ap[row_of(L, s, t) * stride + padl + m] =
            m >= ch.need2[s * L + i] ? min(ch.P[s * L + i] + best, DINF) : DINF;
    }
}

hipError_t launch_fill(const DevChain &ch, const Tables &tb, hipStream_t stream, int32_t *launches,
                       Profiler *prof)
{
    hipError_t e;
    int32_t n = 0;
    if ((e = prof->before(KFILL_INIT)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_init_inf_rows, dim3((tb.stride + 255) / 256), dim3(256), 0, stream, tb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = prof->after()) != hipSuccess) return e;
    ++n;
    const int32_t fin_x = (max(tb.W, tb.padl) + 255) / 256;
    for (int32_t d = 0; d < ch.L; ++d) {
        if (d > 0 && d % BAND == 0) {
            const dim3 grid(((tb.W + 63) / 64) * ((ch.L - d + 15) / 16));
            if ((e = prof->before(KFILL_PRODUCT)) != hipSuccess) return e;
            hipLaunchKernelGGL((k_product<BAND>), grid, dim3(256), 0, stream, ch, tb, d,
                               (int32_t)(tb.max_x <= tb.padl));
            if ((e = hipGetLastError()) != hipSuccess) return e;
            if ((e = prof->after()) != hipSuccess) return e;
            ++n;
            // splits with both operands shorter than d: 2d - d' of them for a cell of span d'
            for (int32_t dd = d; dd < min(d + BAND, ch.L); ++dd)
                prof->work[KFILL_PRODUCT] += (int64_t)(ch.L - dd) * (2 * d - dd) * tb.W;
        }
        if ((e = prof->before(KFILL_FINALIZE)) != hipSuccess) return e;
        hipLaunchKernelGGL(k_finalize, dim3(fin_x * (ch.L - d)), dim3(256), 0, stream, ch, tb, d);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = prof->after()) != hipSuccess) return e;
        ++n;
        const int32_t D = (d / BAND) * BAND;
        prof->work[KFILL_FINALIZE] += (int64_t)(ch.L - d) * ((D > 0 ? 2 * (d - D) : d) + ch.K) * tb.W;
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

// One row of choice codes: thread m scans the candidates in code order.
__global__ __launch_bounds__(256) void k_arg_row(DevChain ch, Tables tb, int32_t s, int32_t t,
                                                 int16_t *__restrict__ out)
{
    const int32_t m = blockIdx.x * 256 + threadIdx.x;
    if (m >= tb.W) return;
    uint64_t best = ~0ull;
    for (int32_t i = s + 1; i <= t; ++i) best = min(best, split_key(ch, tb, s, t, m, i));
    for (int32_t o = 0; o < ch.K; ++o) best = min(best, option_key(ch, tb, s, t, m, o));
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

__device__ inline uint64_t wave_min_u64(uint64_t v)
{
    for (int off = 32; off > 0; off >>= 1) v = min(v, (uint64_t)__shfl_xor((unsigned long long)v, off, 64));
    return v;
}

__global__ __launch_bounds__(64) void k_backtrace(DevChain ch, Tables tb, int32_t m_top,
                                                  rk_op *__restrict__ ops, int64_t cap,
                                                  int64_t *__restrict__ res)
{
    extern __shared__ Frame stk[];
    const int32_t lane = threadIdx.x, L = ch.L, K = ch.K;
    const int32_t stack_cap = 2 * L + 8;
    int32_t sp = 0;
    int64_t n = 0, nfwd = -1, status = 0;

    auto emit = [&](int32_t kind, int32_t block, int32_t option) {
        if (kind == RK_BWD && nfwd < 0) nfwd = n;
        if (lane == 0 && n < cap) ops[n] = rk_op{kind, block, option};
        ++n;
    };
    auto push = [&](Frame f) { stk[sp] = f; ++sp; };

    push(Frame{0, 0, L - 1, m_top});
    while (sp > 0) {
        const Frame f = stk[--sp];
        if (f.type == 1) { emit(f.a, f.b, f.c); continue; }
        const int32_t s = f.a, t = f.b, m = f.c, d = t - s;
        uint64_t key = ~0ull;
        for (int32_t j = lane; j < d + K; j += 64)
            key = min(key, j < d ? split_key(ch, tb, s, t, m, s + 1 + j)
                                 : option_key(ch, tb, s, t, m, j - d));
        key = wave_min_u64(key);
        if (key == ~0ull) { status = 1; break; }
        if ((int32_t)(key >> 32) != opt_at(tb, L, s, t, m)) { status = 2; break; }
        if (sp + 3 > stack_cap) { status = 3; break; }
        const int32_t code = (int32_t)(key & 0xffffffffu);
        if (code >= L) {
            const int32_t o = code - L;
            emit(RK_FWD_SAVE, s, o);
            push(Frame{1, RK_BWD, s, o});
            if (t > s) push(Frame{0, s + 1, t, m - ch.xbar[s * K + o]});
        } else {
            const int32_t i = code;
            emit(RK_FWD_NOSAVE, s, -1);
            for (int32_t k = s + 1; k < i; ++k) {
                emit(RK_FWD_NOSAVE, k, -1);
                emit(RK_FREE_X, k, -1);
            }
            push(Frame{0, s, i - 1, m});
            push(Frame{1, RK_FREE_X, i, -1});
            push(Frame{0, i, t, m - ch.x[i]});
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
    const size_t lds = sizeof(Frame) * (size_t)(2 * ch.L + 8);
    hipLaunchKernelGGL(k_backtrace, dim3(1), dim3(64), lds, stream, ch, tb, m_top, ops, cap, res);
    return hipGetLastError();
}

}  // namespace rk
