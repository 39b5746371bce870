/*
 * rko.h -- CPU oracle of the rk-Rotor dynamic program (Rockmate, App. C).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the plain, slow, single-threaded
 * reference that the HIP path is checked against.  Only the test suite, the
 * package smoke check and the CPU-baseline leg of the benchmark may load it.
 * It shares no code, header, table or helper with the HIP library; the two see
 * the same input arrays and nothing else.
 *
 * Conventions (readings of App. C, stated once here):
 *   - blocks 0..L-1, activations x_0..x_L (x_L is the chain output);
 *   - spans are inclusive: Opt(s,t,m) covers blocks s..t (t >= s);
 *   - m counts every slot the span occupies beyond its own input x_s, which
 *     stays live throughout; the top-level answer is Opt(0, L-1, M - x_0);
 *   - budget columns m = 0..M;
 *   - "infinity" is RKO_INF; every sum saturates there;
 *   - the recorded choice is the lexicographic minimum of (cost, code), with
 *     code = i for the case-2 split that keeps x_i, and code = L + o for the
 *     case-1 option o; -1 where Opt is infinite.
 */
#ifndef RKO_H
#define RKO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RKO_INF INT32_MAX

enum { RKO_FWD_NOSAVE = 0, RKO_FWD_SAVE = 1, RKO_BWD = 2, RKO_FREE_X = 3 };
enum { RKO_OK = 0, RKO_E_INVAL = -1, RKO_E_INFEASIBLE = -6, RKO_E_BUFSZ = -7, RKO_E_REPLAY = -8 };

typedef struct { int32_t kind, block, option; } rko_op;

/* The per-block option sets (App. C notation).  All arrays are row-major,
 * option index fastest: fwd[i*K + o] = r(F_i^o) etc.  fn_* describe F_i^0. */
typedef struct {
    int32_t L, K;
    const int32_t *x;        /* [L+1] */
    const int32_t *fn_time;  /* [L]   r(F_i^0) */
    const int32_t *fn_tmp;   /* [L]   tmp(F_i^0) */
    const int32_t *fwd;      /* [L*K] r(F_i^o) */
    const int32_t *bwd;      /* [L*K] r(B_i^o) */
    const int32_t *mem;      /* [L*K] intermediates kept by F_i^o until B_i^o */
    const int32_t *tmp_fwd;  /* [L*K] tmp(F_i^o) */
    const int32_t *tmp_bwd;  /* [L*K] tmp(B_i^o) */
} rko_chain;

/* Number of spans L(L+1)/2 and the index of span (s,t) in the oracle tables
 * (upper triangle, row-major in s). */
int64_t rko_ncells(int32_t L);
int64_t rko_cell(int32_t L, int32_t s, int32_t t);

/* Fill Opt and the choice table for every span and every m in [0, M]
 * (Eqs. fe, fn and all; Alg. 2).  Tables are m-major:
 *   opt[m * ncells + cell(s,t)], arg[m * ncells + cell(s,t)].
 * *answer = Opt(0, L-1, M - x_0), or RKO_INF when infeasible or M < x_0. */
int rko_solve(const rko_chain *c, int32_t M, int32_t *opt, int16_t *arg, int32_t *answer);

/* Alg. 3 over the choice table, for budget M, with the forgets of x_k made
 * explicit.  Two-call: if ops is NULL or cap is too small, *n_ops receives
 * the length and RKO_E_BUFSZ is returned.  *n_fwd = index of the first
 * backward (the forward/backward split of the schedule). */
int rko_schedule(const rko_chain *c, int32_t M, const int16_t *arg, rko_op *ops, int64_t cap,
                 int64_t *n_ops, int64_t *n_fwd);

/* Replay a schedule from the state {x_0 live} and check that it ends with
 * every backward done and only x_0 live.  Memory follows App. C: running
 * F_k^0 needs its input, its output and tmp(F_k^0); F_k^o additionally keeps
 * its intermediates until B_k^o, which needs tmp(B_k^o) on top.
 * Returns RKO_OK or RKO_E_REPLAY (with *bad = index of the first illegal op,
 * or n for a wrong final state). */
int rko_simulate(const rko_chain *c, const rko_op *ops, int64_t n, int64_t *time, int64_t *peak,
                 int64_t *bad);

/* Smallest budget m (beyond x_s) at which span (s,t) has any valid schedule,
 * by a recursion over spans with no budget axis.  out[cell(s,t)]. */
int rko_min_feasible(const rko_chain *c, int64_t *out);

#ifdef __cplusplus
}
#endif
#endif
