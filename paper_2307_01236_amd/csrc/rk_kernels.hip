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
// Band product.  For the spans d in [tau, tau + T) (one band), the part of Eq. fn over
// the splits i whose two operands are older than the band: both s..i-1 and i..t shorter
// than tau.  That is a min-plus product
//     acc(s,t) = min_i ap(s,i) + Opt(i, t, m - x_i)
// elementwise in m.  A wavefront owns 64 consecutive budgets (lane = m) and SR rows s;
// each of its lanes keeps SR x T accumulators, so every loaded ap value is used T times
// and every loaded Opt value up to SR times.  Operands outside the window (not final
// yet, or not a span) are read from the infinity row, which keeps the loop free of masks.
// The partial minimum goes into the Opt slot of each cell; the finalize kernel of its
// diagonal completes it.
// ---------------------------------------------------------------------------------------
template <int T, int SR>
__global__ __launch_bounds__(256) void k_product(DevChain ch, Tables tb, int32_t tau)
{
    const int32_t L = ch.L;
    const int32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int32_t m = blockIdx.x * 64 + lane;
    const int32_t s0 = (blockIdx.y * 4 + wave) * SR;
    const int32_t s_end = L - tau;  // rows that own at least one cell of the band
    if (s0 >= s_end) return;
    const int64_t stride = tb.stride;
    const int32_t col = tb.padl + min(m, tb.W - 1);
    const int32_t *const inf_a = tb.ap + tb.inf_row * stride + col;
    const int32_t *const inf_q = tb.opt + tb.inf_row * stride + col;

    int32_t acc[SR][T];
#pragma unroll
    for (int r = 0; r < SR; ++r)
#pragma unroll
        for (int k = 0; k < T; ++k) acc[r][k] = DINF;

    const int32_t i_lo = s0 + 1;
    const int32_t i_hi = min(s0 + SR - 1 + tau, L - 1);
    for (int32_t i = i_lo; i <= i_hi; ++i) {
        int32_t a[SR];
#pragma unroll
        for (int r = 0; r < SR; ++r) {
            const int32_t s = s0 + r, span = i - 1 - s;
            const bool ok = s < s_end && span >= 0 && span < tau;
            a[r] = ok ? tb.ap[row_of(L, s, i - 1) * stride + col] : *inf_a;
        }
        const int32_t xi = ch.x[i];
        const bool xok = xi <= tb.padl;
        int32_t q[SR + T - 1];
#pragma unroll
        for (int j = 0; j < SR + T - 1; ++j) {
            const int32_t t = s0 + tau + j, span = t - i;
            const bool ok = xok && t < L && span >= 0 && span < tau;
            q[j] = ok ? tb.opt[row_of(L, i, t) * stride + (col - xi)] : *inf_q;
        }
#pragma unroll
        for (int r = 0; r < SR; ++r)
#pragma unroll
            for (int k = 0; k < T; ++k) acc[r][k] = min(acc[r][k], a[r] + q[r + k]);
    }
    if (m >= tb.W) return;
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
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_finalize(DevChain ch, Tables tb, int32_t d)
{
    const int32_t s = blockIdx.y, L = ch.L, K = ch.K, t = s + d;
    const int32_t m = blockIdx.x * 256 + threadIdx.x;
    const int64_t stride = tb.stride;
    const int64_t row = row_of(L, s, t) * stride;
    if (m < tb.padl) tb.opt[row + m] = DINF;  // keep the left pad infinite
    if (m >= tb.W) return;
    const int32_t col = tb.padl + m;
    const int32_t D = (d / BAND) * BAND;
    int32_t best = D > 0 ? tb.opt[row + col] : DINF;

    auto split = [&](int32_t i) {
        const int32_t a = tb.ap[row_of(L, s, i - 1) * stride + col];
        const int32_t xi = ch.x[i];
        const int32_t q = xi <= tb.padl ? tb.opt[row_of(L, i, t) * stride + (col - xi)] : DINF;
        best = min(best, a + q);
    };
    if (D == 0) {
        for (int32_t i = s + 1; i <= t; ++i) split(i);
    } else {
        for (int32_t i = s + 1; i <= t - D; ++i) split(i);      // t - i >= D
        for (int32_t i = s + D + 1; i <= t; ++i) split(i);      // i - 1 - s >= D
    }
    // case 1, option o: r(F_s^o) + r(B_s^o) + Opt(s+1,t,m-xbar), valid iff m >= need1[s][o]
    const int64_t rest_row = d > 0 ? row_of(L, s + 1, t) * stride + tb.padl : 0;
    for (int32_t o = 0; o < K; ++o) {
        if (m >= ch.need1[s * K + o]) {
            const int32_t rest = d > 0 ? tb.opt[rest_row + (m - ch.xbar[s * K + o])] : 0;
            best = min(best, ch.c1[s * K + o] + rest);
        }
    }
    best = min(best, DINF);
    tb.opt[row + col] = best;
    if (t + 1 < L) {
        const int32_t i = t + 1;
        tb.ap[row + col] = m >= ch.need2[s * L + i] ? min(ch.P[s * L + i] + best, DINF) : DINF;
    }
}

hipError_t launch_fill(const DevChain &ch, const Tables &tb, hipStream_t stream, int32_t *launches,
                       Profiler *prof)
{
    constexpr int SR = 4;
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
            const dim3 grid((tb.W + 63) / 64, (ch.L - d + 4 * SR - 1) / (4 * SR));
            if ((e = prof->before(KFILL_PRODUCT)) != hipSuccess) return e;
            hipLaunchKernelGGL((k_product<BAND, SR>), grid, dim3(256), 0, stream, ch, tb, d);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            if ((e = prof->after()) != hipSuccess) return e;
            ++n;
            // splits with both operands shorter than d: 2d - d' of them for a cell of span d'
            for (int32_t dd = d; dd < min(d + BAND, ch.L); ++dd)
                prof->work[KFILL_PRODUCT] += (int64_t)(ch.L - dd) * (2 * d - dd) * tb.W;
        }
        if ((e = prof->before(KFILL_FINALIZE)) != hipSuccess) return e;
        hipLaunchKernelGGL(k_finalize, dim3(fin_x, ch.L - d), dim3(256), 0, stream, ch, tb, d);
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
