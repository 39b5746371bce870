// rk_host.h -- host-side derivation of a chain's per-block, per-option and per-span
// quantities (App. C notation), in plain C++ with no HIP dependency, so that it also
// builds on its own (the sanitizer test compiles it with g++).
#pragma once

#include <stdint.h>

#include <vector>

#include "rk.h"

namespace rk {

struct HostChain {
    int32_t L = 0, K = 0;
    std::vector<int32_t> x, fn_time, fn_tmp;  // [L+1], [L], [L]
    std::vector<int32_t> xbar, c1, need1, mem;  // [L*K]: x_{s+1} + mem, r(F)+r(B), case 1's need, mem
    std::vector<int32_t> P, need2;              // [L*L]: sweep time and need of case 2 (s < i)
    // From budget msa(s,t) on, storing everything fits and Opt(s,t,m) = lb(s,t); [L(L+1)/2]
    // in upper-triangle row-major order (row(s,t) = sL - s(s-1)/2 + t - s)
    std::vector<int32_t> msa, lb;
    std::vector<int64_t> fmax, bmax;  // [L]: largest forward time (any kind) and backward time
    // The saving sweep (empty when off): refwd, c3 = r(F)+r(B)+refwd [L*K]; need3[s*L+i] =
    // max_{k=s}^{i-1} x_k + x_{k+1} + tmp(F_k^0), the sweep of H(s, .) that drops its input
    std::vector<int32_t> refwd, c3, need3;
    // From budget msaH(s,t) on (t > s), H(s,t,u) = lb(s,t) + P[s][s+1]: every candidate of H
    // is at least lb(s,t) + P[s][i] >= lb(s,t) + P[s][s+1], and split s+1 reaches it once its
    // sweep fits (need3[s][s+1] <= u) and both of its parts are past their msa
    // (u - x_s >= msa(s,s), u - x_{s+1} >= msa(s+1,t)); [L(L+1)/2] like msa
    std::vector<int32_t> msaH;
    std::vector<uint8_t> kept;  // [L*K] option survives the dominance test
    int32_t max_x = 0;          // largest x_i over the split points i = 1..L-1
};

// Checks the inputs (see rk_chain_create) and derives everything but the saving sweep.
// Returns RK_OK, RK_E_INVAL or RK_E_OVERFLOW; throws std::bad_alloc when out of memory.
int host_create(HostChain &h, int32_t L, int32_t K, const int32_t *x, const int32_t *fn_time,
                const int32_t *fn_tmp, const int32_t *fwd, const int32_t *bwd, const int32_t *mem,
                const int32_t *tmp_fwd, const int32_t *tmp_bwd);

// Switches the saving sweep on with these re-forward times ([L*K]) or off (NULL), and
// redoes the dominance test.  RK_E_INVAL for a negative time or L + 2K >= 32768 (choice
// codes), RK_E_OVERFLOW when schedule times could pass RK_TIME_LIMIT; the chain is left
// unchanged then.
int host_set_refwd(HostChain &h, const int32_t *refwd);

// The option slots the kernels evaluate: per block the kept options (every option when
// prune is false) in the caller's order, padded to k_run slots with slots that never win.
struct RunSlots {
    int32_t k_run = 0;
    std::vector<int32_t> opt;  // [L*k_run] caller's option index, -1 for padding
    std::vector<int32_t> xbar, c1, need1, c3;  // [L*k_run] (c3 empty without the sweep)
    std::vector<int32_t> need1max;             // [L]
};
void host_run_slots(const HostChain &h, bool prune, RunSlots &r);

}  // namespace rk
