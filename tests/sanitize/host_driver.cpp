// Drives the host precompute of librkrotor (rk_host.cpp) over many generated chains, for
// a build with AddressSanitizer and UndefinedBehaviorSanitizer: valid chains of many
// shapes (1..300 blocks, 1..40 options, zeros, values near the saturation caps, repeated
// options), invalid ones (negative entries, too many options, time overflow), the saving
// sweep on and off, and the option slots with pruning on and off.  Prints one checksum
// line per chain; exits non-zero on a failed invariant.
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "rk_host.h"

namespace {

uint64_t state = 0x9e3779b97f4a7c15ull;
uint32_t next()
{
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return (uint32_t)(state >> 11);
}
int32_t pick(int32_t lo, int32_t hi) { return lo + (int32_t)(next() % (uint32_t)(hi - lo + 1)); }

int fail(const char *what, int k)
{
    printf("FAIL %s (chain %d)\n", what, k);
    return 1;
}

}  // namespace

int main()
{
    for (int k = 0; k < 400; ++k) {
        const int32_t L = k % 37 == 0 ? 1 : pick(1, k % 50 == 0 ? 300 : 40);
        const int32_t K = k % 29 == 0 ? 1 : pick(1, 40);
        const int32_t big = k % 7 == 0 ? (1 << 29) : 1000;  // sizes near the caps now and then
        const int32_t tmax = k % 11 == 0 ? 0 : 50;
        std::vector<int32_t> x(L + 1), fn(L), fnt(L), fwd(L * K), bwd(L * K), mem(L * K), tf(L * K), tb(L * K);
        for (auto &v : x) v = pick(0, k % 7 == 0 ? big : 20);
        for (int32_t i = 0; i < L; ++i) {
            fn[i] = pick(0, 100);
            fnt[i] = pick(0, tmax);
            for (int32_t o = 0; o < K; ++o) {
                const int32_t j = i * K + o;
                const bool rep = o > 0 && next() % 4 == 0;  // a repeated option
                fwd[j] = rep ? fwd[j - 1] : pick(0, 100);
                bwd[j] = rep ? bwd[j - 1] : pick(0, 200);
                mem[j] = rep ? mem[j - 1] : pick(0, k % 7 == 0 ? big : 60);
                tf[j] = rep ? tf[j - 1] : pick(0, tmax);
                tb[j] = rep ? tb[j - 1] : pick(0, tmax);
            }
        }
        if (k % 13 == 5) mem[next() % (L * K)] = -1;                // invalid
        if (k % 17 == 3) fwd[next() % (L * K)] = 1 << 30;           // time overflow
        rk::HostChain h;
        const int rc = rk::host_create(h, L, K, x.data(), fn.data(), fnt.data(), fwd.data(), bwd.data(), mem.data(),
                                       tf.data(), tb.data());
        if (k % 13 == 5 && rc != RK_E_INVAL) return fail("negative size accepted", k);
        if (k % 17 == 3 && k % 13 != 5 && rc != RK_E_OVERFLOW) return fail("time overflow accepted", k);
        if (rc != RK_OK) {
            printf("%d rc %d\n", k, rc);
            continue;
        }
        uint64_t sum = 0;
        for (int sweep = 0; sweep < 2; ++sweep) {
            std::vector<int32_t> refwd(L * K);
            for (auto &v : refwd) v = pick(0, 150);
            const int rs = rk::host_set_refwd(h, sweep ? refwd.data() : nullptr);
            if (rs != RK_OK) return fail("host_set_refwd", k);
            for (int prune = 0; prune < 2; ++prune) {
                rk::RunSlots r;
                rk::host_run_slots(h, prune != 0, r);
                if (r.k_run < 1 || r.k_run > K) return fail("k_run", k);
                if ((int)r.opt.size() != L * r.k_run) return fail("slots", k);
                for (int32_t s = 0; s < L; ++s)
                    for (int32_t q = 0; q < r.k_run; ++q) {
                        const int32_t o = r.opt[s * r.k_run + q];
                        if (o >= 0 && r.need1[s * r.k_run + q] > r.need1max[s]) return fail("need1max", k);
                        sum = sum * 31 + (uint32_t)(o + 1) + (uint32_t)r.xbar[s * r.k_run + q];
                    }
            }
        }
        for (int32_t t = 0; t < L; ++t)
            for (int32_t s = 0; s <= t; ++s) {
                const int64_t row = (int64_t)s * L - (int64_t)s * (s - 1) / 2 + (t - s);
                if (h.msa[row] < 0 || h.lb[row] < 0) return fail("msa/lb sign", k);
                // a longer span needs at least the memory and time of the shorter one
                if (t > s && (h.msa[row] < h.msa[row - 1] || h.lb[row] < h.lb[row - 1])) return fail("monotone", k);
                sum = sum * 31 + (uint32_t)h.msa[row] + (uint32_t)h.lb[row];
            }
        printf("%d ok %llu\n", k, (unsigned long long)sum);
    }
    return 0;
}
