// rk_host.cpp -- the per-chain precompute of rk_chain_create (App. C quantities), the
// dominance test on options and the option slots of the kernels.  Plain C++.
#include "rk_host.h"

#include <algorithm>

namespace rk {

namespace {

constexpr int64_t kSizeCap = int64_t(1) << 30;  // derived sizes saturate here (above any budget)
constexpr int32_t kDinf = (1 << 30) - 1;        // the kernels' infinity

int64_t row(int32_t L, int32_t s, int32_t t) { return (int64_t)s * L - (int64_t)s * (s - 1) / 2 + (t - s); }

// Schedule-time bound: a block is forwarded at most L times (any forward kind, the
// re-forward of the saving sweep included) and backwarded once.
bool time_fits(const HostChain &h, const int32_t *refwd)
{
    int64_t fsum = 0, bsum = 0;
    for (int32_t i = 0; i < h.L; ++i) {
        int64_t f = h.fmax[i];
        if (refwd)
            for (int32_t o = 0; o < h.K; ++o) f = std::max<int64_t>(f, refwd[(int64_t)i * h.K + o]);
        fsum += f;
        bsum += h.bmax[i];
    }
    return (int64_t)h.L * fsum + bsum <= RK_TIME_LIMIT;
}

// Option o of block s is never the recorded choice when an earlier option o' < o of the
// block is at least as good in all that Eq. fe reads: r(F)+r(B), xbar and the memory the
// pair needs (and, with the saving sweep, its cost c3; mem follows from xbar).  Then o' is a
// candidate wherever o is, and (Opt and H being non-increasing in m) never costs more; at
// equal cost it wins by its smaller code.  Testing against the kept options suffices:
// dominance is transitive.  This also drops repeated options, which the paper's budget
// grid produces many of (Sec. 3, Phase 2).
void prune(HostChain &h)
{
    const int32_t L = h.L, K = h.K;
    const bool sweep = !h.refwd.empty();
    h.kept.assign((size_t)L * K, 1);
    for (int32_t s = 0; s < L; ++s)
        for (int32_t o = 1; o < K; ++o) {
            const size_t j = (size_t)s * K + o;
            for (int32_t q = 0; q < o; ++q) {
                const size_t i = (size_t)s * K + q;
                if (h.kept[i] && h.c1[i] <= h.c1[j] && h.xbar[i] <= h.xbar[j] && h.need1[i] <= h.need1[j] &&
                    (!sweep || h.c3[i] <= h.c3[j])) {
                    h.kept[j] = 0;
                    break;
                }
            }
        }
}

}  // namespace

int host_create(HostChain &h, int32_t L, int32_t K, const int32_t *x, const int32_t *fn_time,
                const int32_t *fn_tmp, const int32_t *fwd, const int32_t *bwd, const int32_t *mem,
                const int32_t *tmp_fwd, const int32_t *tmp_bwd)
{
    if (L < 1 || L > RK_MAX_L || K < 1 || (int64_t)L + K >= 32768) return RK_E_INVAL;
    if (!x || !fn_time || !fn_tmp || !fwd || !bwd || !mem || !tmp_fwd || !tmp_bwd) return RK_E_INVAL;
    const int64_t nk = (int64_t)L * K;
    for (int32_t i = 0; i <= L; ++i)
        if (x[i] < 0) return RK_E_INVAL;
    for (int32_t i = 0; i < L; ++i)
        if (fn_time[i] < 0 || fn_tmp[i] < 0) return RK_E_INVAL;
    for (int64_t j = 0; j < nk; ++j)
        if (fwd[j] < 0 || bwd[j] < 0 || mem[j] < 0 || tmp_fwd[j] < 0 || tmp_bwd[j] < 0) return RK_E_INVAL;

    h.L = L;
    h.K = K;
    h.fmax.assign(L, 0);
    h.bmax.assign(L, 0);
    for (int32_t i = 0; i < L; ++i) {
        int64_t fm = fn_time[i], bm = 0;
        for (int32_t o = 0; o < K; ++o) {
            fm = std::max<int64_t>(fm, fwd[(int64_t)i * K + o]);
            bm = std::max<int64_t>(bm, bwd[(int64_t)i * K + o]);
        }
        h.fmax[i] = fm;
        h.bmax[i] = bm;
    }
    if (!time_fits(h, nullptr)) return RK_E_OVERFLOW;

    h.x.assign(x, x + L + 1);
    h.fn_time.assign(fn_time, fn_time + L);
    h.fn_tmp.assign(fn_tmp, fn_tmp + L);
    h.xbar.resize(nk);
    h.c1.resize(nk);
    h.need1.resize(nk);
    h.mem.assign(mem, mem + nk);
    h.refwd.clear();
    h.c3.clear();
    h.need3.clear();
    // Case 1 (Eq. fe): F_s^o leaves xbar = x_{s+1} + mem live; it and B_s^o need their
    // temporary memory on top of that; the pair costs r(F_s^o) + r(B_s^o).
    for (int32_t s = 0; s < L; ++s)
        for (int32_t o = 0; o < K; ++o) {
            const int64_t j = (int64_t)s * K + o;
            const int64_t xb = (int64_t)x[s + 1] + mem[j];
            h.xbar[j] = (int32_t)std::min(xb, kSizeCap);
            h.need1[j] = (int32_t)std::min(xb + std::max(tmp_fwd[j], tmp_bwd[j]), kSizeCap);
            h.c1[j] = fwd[j] + bwd[j];
        }
    prune(h);
    // Case 2 (Eq. fn): the sweep F_s^0..F_{i-1}^0 costs P[s][i]; F_k^0 holds its input
    // (except the span input x_s, outside the budget), its output and tmp(F_k^0).
    h.P.assign((size_t)L * L, 0);
    h.need2.assign((size_t)L * L, 0);
    for (int32_t s = 0; s < L; ++s) {
        int64_t p = 0, need = 0;
        for (int32_t i = s + 1; i < L; ++i) {
            const int32_t k = i - 1;
            p += fn_time[k];
            need = std::max<int64_t>(need, (k > s ? (int64_t)x[k] : 0) + x[k + 1] + fn_tmp[k]);
            h.P[(size_t)s * L + i] = (int32_t)p;
            h.need2[(size_t)s * L + i] = (int32_t)std::min(need, kSizeCap);
        }
    }
    // Storing everything: every schedule of a span runs each of its blocks' backward once,
    // paired with one saving forward, so it costs at least lb(s,t) = sum of min_o r(F)+r(B)
    // (further forwards, re-forwards included, only add).  Case 1 with a cheapest option at
    // every block reaches lb as soon as it fits, from msa(s,t) = min over the cheapest
    // options o of block s of max(need1[s][o], xbar[s][o] + msa(s+1,t)) (msa(s,s): the
    // smallest need1).  Opt being non-increasing in m, Opt(s,t,m) = lb(s,t) for m >= msa(s,t).
    const size_t nr = (size_t)L * (L + 1) / 2;
    h.msa.assign(nr, 0);
    h.lb.assign(nr, 0);
    std::vector<int64_t> cmin(L), prefix(L + 1, 0);
    for (int32_t s = 0; s < L; ++s) {
        int64_t v = INT64_MAX;
        for (int32_t o = 0; o < K; ++o) v = std::min<int64_t>(v, h.c1[(size_t)s * K + o]);
        cmin[s] = v;
        prefix[s + 1] = prefix[s] + v;
    }
    for (int32_t t = 0; t < L; ++t)
        for (int32_t s = t; s >= 0; --s) {
            const int64_t rest = s < t ? h.msa[(size_t)row(L, s + 1, t)] : 0;
            int64_t best = kSizeCap;
            for (int32_t o = 0; o < K; ++o) {
                const size_t j = (size_t)s * K + o;
                if (h.c1[j] != cmin[s]) continue;
                best = std::min(best, std::max<int64_t>(h.need1[j], s < t ? h.xbar[j] + rest : 0));
            }
            h.msa[(size_t)row(L, s, t)] = (int32_t)std::min(best, kSizeCap);
            h.lb[(size_t)row(L, s, t)] = (int32_t)(prefix[t + 1] - prefix[s]);
        }
    h.max_x = 0;
    for (int32_t i = 1; i < L; ++i) h.max_x = std::max(h.max_x, x[i]);
    return RK_OK;
}

int host_set_refwd(HostChain &h, const int32_t *refwd)
{
    const int32_t L = h.L, K = h.K;
    if (!refwd) {
        h.refwd.clear();
        h.c3.clear();
        h.need3.clear();
        h.msaH.clear();
        prune(h);
        return RK_OK;
    }
    if ((int64_t)L + 2 * (int64_t)K >= 32768) return RK_E_INVAL;
    const int64_t nk = (int64_t)L * K;
    for (int64_t j = 0; j < nk; ++j)
        if (refwd[j] < 0) return RK_E_INVAL;
    if (!time_fits(h, refwd)) return RK_E_OVERFLOW;
    h.refwd.assign(refwd, refwd + nk);
    h.c3.resize(nk);
    for (int64_t j = 0; j < nk; ++j) h.c3[j] = (int32_t)std::min<int64_t>((int64_t)h.c1[j] + refwd[j], kSizeCap);
    // The sweep of H(s, t): F_s^0..F_{i-1}^0 with every input inside the budget (the input
    // x_s is dropped too, and made again later from the data block s-1 kept).
    h.need3.assign((size_t)L * L, 0);
    for (int32_t s = 0; s < L; ++s) {
        int64_t need = 0;
        for (int32_t i = s + 1; i < L; ++i) {
            const int32_t k = i - 1;
            need = std::max<int64_t>(need, (int64_t)h.x[k] + h.x[k + 1] + h.fn_tmp[k]);
            h.need3[(size_t)s * L + i] = (int32_t)std::min(need, kSizeCap);
        }
    }
    h.msaH.assign(h.msa.size(), (int32_t)kSizeCap);
    for (int32_t s = 0; s + 1 < L; ++s)
        for (int32_t t = s + 1; t < L; ++t) {
            const int64_t v = std::max<int64_t>({h.need3[(size_t)s * L + s + 1],
                                                 (int64_t)h.msa[(size_t)row(L, s, s)] + h.x[s],
                                                 (int64_t)h.msa[(size_t)row(L, s + 1, t)] + h.x[s + 1]});
            h.msaH[(size_t)row(L, s, t)] = (int32_t)std::min(v, kSizeCap);
        }
    prune(h);
    return RK_OK;
}

// A padding slot costs the device infinity and needs only x_{s+1}: wherever it is a
// candidate its value is at or above infinity, so it never changes a minimum and is never
// the recorded choice.
void host_run_slots(const HostChain &h, bool prune_on, RunSlots &r)
{
    const int32_t L = h.L, K = h.K;
    const bool sweep = !h.refwd.empty();
    int32_t kr = 1;
    for (int32_t s = 0; s < L; ++s) {
        int32_t n = 0;
        for (int32_t o = 0; o < K; ++o) n += !prune_on || h.kept[(size_t)s * K + o];
        kr = std::max(kr, n);
    }
    r.k_run = kr;
    const size_t nr = (size_t)L * kr;
    r.opt.assign(nr, -1);
    r.xbar.assign(nr, 0);
    r.c1.assign(nr, kDinf);
    r.need1.assign(nr, 0);
    if (sweep) r.c3.assign(nr, kDinf);
    else r.c3.clear();
    r.need1max.assign(L, 0);
    for (int32_t s = 0; s < L; ++s) {
        int32_t slot = 0;
        for (int32_t o = 0; o < K; ++o) {
            const size_t j = (size_t)s * K + o;
            if (prune_on && !h.kept[j]) continue;
            const size_t q = (size_t)s * kr + slot++;
            r.opt[q] = o;
            r.xbar[q] = h.xbar[j];
            r.c1[q] = h.c1[j];
            r.need1[q] = h.need1[j];
            if (sweep) r.c3[q] = h.c3[j];
            r.need1max[s] = std::max(r.need1max[s], h.need1[j]);
        }
        for (; slot < kr; ++slot) {
            const size_t q = (size_t)s * kr + slot;
            r.xbar[q] = r.need1[q] = h.x[s + 1];
        }
    }
}

}  // namespace rk
