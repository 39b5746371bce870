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

// ---------------------------------------------------------------------------------------
// Fill of one span-length diagonal d: thread (s, m).
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_fill_diag(DevChain ch, int32_t *__restrict__ tab,
                                                   int32_t W, int32_t stride, int32_t d)
{
    const int32_t s = blockIdx.y;
    const int32_t m = blockIdx.x * 256 + threadIdx.x;
    if (m >= W) return;
    const int32_t L = ch.L, K = ch.K, t = s + d;
    int32_t best = DINF;
    if (d > 0) {
        // case 2, split i: P[s][i] + Opt(s,i-1,m) + Opt(i,t,m-x_i), valid iff m >= need2[s][i]
        for (int32_t i = s + 1; i <= t; ++i) {
            if (m >= ch.need2[s * L + i]) {
                const int32_t a = tab[row_of(L, s, i - 1) * stride + m];
                const int32_t q = tab[row_of(L, i, t) * stride + (m - ch.x[i])];
                best = min(best, min(ch.P[s * L + i] + a, DINF) + q);
            }
        }
    }
    // case 1, option o: r(F_s^o) + r(B_s^o) + Opt(s+1,t,m-xbar), valid iff m >= need1[s][o]
    const int64_t rest_row = d > 0 ? row_of(L, s + 1, t) * stride : 0;
    for (int32_t o = 0; o < K; ++o) {
        if (m >= ch.need1[s * K + o]) {
            const int32_t rest = d > 0 ? tab[rest_row + (m - ch.xbar[s * K + o])] : 0;
            best = min(best, ch.c1[s * K + o] + rest);
        }
    }
    tab[row_of(L, s, t) * stride + m] = min(best, DINF);
}

const char *const kFillKernelNames[KFILL_NKINDS] = {"k_fill_diag"};

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

hipError_t launch_fill(const DevChain &ch, int32_t *tab, int32_t W, int32_t stride,
                       hipStream_t stream, int32_t *launches, Profiler *prof)
{
    const dim3 block(256);
    hipError_t e;
    for (int32_t d = 0; d < ch.L; ++d) {
        const dim3 grid((W + 255) / 256, ch.L - d);
        if ((e = prof->before(KFILL_DIAG)) != hipSuccess) return e;
        hipLaunchKernelGGL(k_fill_diag, grid, block, 0, stream, ch, tab, W, stride, d);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = prof->after()) != hipSuccess) return e;
    }
    *launches = ch.L;
    return hipSuccess;
}

// ---------------------------------------------------------------------------------------
// Choice recovery.  The key of a candidate is (cost << 32) | code, so the smallest key is
// the lexicographic (cost, code) minimum; invalid or infinite candidates get ~0.
// ---------------------------------------------------------------------------------------
__device__ inline uint64_t split_key(const DevChain &ch, const int32_t *tab, int32_t stride,
                                     int32_t s, int32_t t, int32_t m, int32_t i)
{
    const int32_t L = ch.L;
    if (m < ch.need2[s * L + i]) return ~0ull;
    const int32_t a = tab[row_of(L, s, i - 1) * stride + m];
    const int32_t q = tab[row_of(L, i, t) * stride + (m - ch.x[i])];
    if (a >= DINF || q >= DINF) return ~0ull;
    const int64_t v = (int64_t)ch.P[s * L + i] + a + q;
    if (v >= DINF) return ~0ull;
    return ((uint64_t)v << 32) | (uint32_t)i;
}

__device__ inline uint64_t option_key(const DevChain &ch, const int32_t *tab, int32_t stride,
                                      int32_t s, int32_t t, int32_t m, int32_t o)
{
    const int32_t L = ch.L, K = ch.K;
    if (m < ch.need1[s * K + o]) return ~0ull;
    int32_t rest = 0;
    if (t > s) rest = tab[row_of(L, s + 1, t) * stride + (m - ch.xbar[s * K + o])];
    if (rest >= DINF) return ~0ull;
    const int64_t v = (int64_t)ch.c1[s * K + o] + rest;
    if (v >= DINF) return ~0ull;
    return ((uint64_t)v << 32) | (uint32_t)(L + o);
}

// One row of choice codes: thread m scans the candidates in code order.
__global__ __launch_bounds__(256) void k_arg_row(DevChain ch, const int32_t *__restrict__ tab,
                                                 int32_t W, int32_t stride, int32_t s, int32_t t,
                                                 int16_t *__restrict__ out)
{
    const int32_t m = blockIdx.x * 256 + threadIdx.x;
    if (m >= W) return;
    uint64_t best = ~0ull;
    for (int32_t i = s + 1; i <= t; ++i) best = min(best, split_key(ch, tab, stride, s, t, m, i));
    for (int32_t o = 0; o < ch.K; ++o) best = min(best, option_key(ch, tab, stride, s, t, m, o));
    out[m] = best == ~0ull ? (int16_t)-1 : (int16_t)(best & 0xffffu);
}

hipError_t launch_arg_row(const DevChain &ch, const int32_t *tab, int32_t W, int32_t stride,
                          int32_t s, int32_t t, int16_t *out, hipStream_t stream)
{
    hipLaunchKernelGGL(k_arg_row, dim3((W + 255) / 256), dim3(256), 0, stream, ch, tab, W, stride,
                       s, t, out);
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

__global__ __launch_bounds__(64) void k_backtrace(DevChain ch, const int32_t *__restrict__ tab,
                                                  int32_t stride, int32_t m_top, rk_op *__restrict__ ops,
                                                  int64_t cap, int64_t *__restrict__ res)
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
            key = min(key, j < d ? split_key(ch, tab, stride, s, t, m, s + 1 + j)
                                 : option_key(ch, tab, stride, s, t, m, j - d));
        key = wave_min_u64(key);
        if (key == ~0ull) { status = 1; break; }
        if ((int32_t)(key >> 32) != tab[row_of(L, s, t) * stride + m]) { status = 2; break; }
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

hipError_t launch_backtrace(const DevChain &ch, const int32_t *tab, int32_t stride, int32_t m_top,
                            rk_op *ops, int64_t cap, int64_t *res, hipStream_t stream)
{
    const size_t lds = sizeof(Frame) * (size_t)(2 * ch.L + 8);
    hipLaunchKernelGGL(k_backtrace, dim3(1), dim3(64), lds, stream, ch, tab, stride, m_top, ops, cap,
                       res);
    return hipGetLastError();
}

}  // namespace rk
