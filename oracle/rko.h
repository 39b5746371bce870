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

enum { RKO_FWD_NOSAVE = 0, RKO_FWD_SAVE = 1, RKO_BWD = 2, RKO_FREE_X = 3, RKO_REFWD = 4 };
enum { RKO_OK = 0, RKO_E_INVAL = -1, RKO_E_INFEASIBLE = -6, RKO_E_BUFSZ = -7, RKO_E_REPLAY = -8 };

typedef struct { int32_t kind, block, option; } rko_op;

/* The per-block option sets (App. C notation).  All arrays are row-major,
 * option index fastest: fwd[i*K + o] = r(F_i^o) etc.  fn_* describe F_i^0.
 *
 * refwd (NULL: off) widens case 2 with the saving sweep of the sub-optimality
 * remark (ii) of Sec. 3.4: refwd[i*K + o] is the time to compute x_{i+1} again
 * from the intermediates that F_i^o kept (with tmp(F_i^o) of temporary memory).
 * Case 3 of span (s,t), option o of block s: F_s^o keeps its intermediates,
 * then F_{s+1}^0 .. F_{i-1}^0 sweep to x_i dropping everything behind them
 * (x_{s+1} included), the subproblem i..t runs, x_i is dropped, x_{s+1} is
 * computed again from the kept data (RKO_REFWD), the subproblem s+1..i-1 runs,
 * and B_s^o ends the span:
 *   Opt_3(s,t,m) = min_o r(F_s^o) + r(B_s^o) + refwd + H(s+1, t, m - mem_s^o),
 *   H(s',t,u)   = min_i sum_{k=s'}^{i-1} r(F_k^0) + Opt(i,t,u - x_i) + Opt(s',i-1,u - x_s'),
 * for t >= s+2 and i = s'+1..t, valid when the option is (case 1's test) and
 * every F_k^0 of the sweep fits u with its input, its output and tmp(F_k^0).
 * Its choice code is L + K + o (after case 2's i and case 1's L + o). */
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
    const int32_t *refwd;    /* [L*K] or NULL: time of recomputing x_{i+1} from what F_i^o kept */
} rko_chain;

/* Number of spans L(L+1)/2 and the index of span (s,t) in the oracle tables
 * (upper triangle, row-major in s). */
int64_t rko_ncells(int32_t L);
int64_t rko_cell(int32_t L, int32_t s, int32_t t);

/* Fill Opt and the choice table for every span and every m in [0, M]
 * (Eqs. fe, fn and all; Alg. 2).  Tables are m-major:
 *   opt[m * ncells + cell(s,t)], arg[m * ncells + cell(s,t)].
 * With c->refwd set, hval and harg (same layout) receive H(s,t,u) of the saving
 * sweep and its choice (the split i, -1 where infinite; single blocks: INF, -1);
 * they must then be non-NULL, else they are ignored and may be NULL.
 * *answer = Opt(0, L-1, M - x_0), or RKO_INF when infeasible or M < x_0. */
int rko_solve(const rko_chain *c, int32_t M, int32_t *opt, int16_t *arg, int32_t *hval, int16_t *harg,
              int32_t *answer);

/* Alg. 3 over the choice table, for budget M, with the forgets of x_k made
 * explicit (and, with refwd, case 3 laid out as described above, its split
 * read from harg).  Two-call: if ops is NULL or cap is too small, *n_ops
 * receives the length and RKO_E_BUFSZ is returned.  *n_fwd = index of the
 * first backward (the forward/backward split of the schedule). */
int rko_schedule(const rko_chain *c, int32_t M, const int16_t *arg, const int16_t *harg, rko_op *ops,
                 int64_t cap, int64_t *n_ops, int64_t *n_fwd);

/* Replay a schedule from the state {x_0 live} and check that it ends with
 * every backward done and only x_0 live.  Memory follows App. C: running
 * F_k^0 needs its input, its output and tmp(F_k^0); F_k^o additionally keeps
 * its intermediates until B_k^o, which needs tmp(B_k^o) on top; RKO_REFWD
 * (needs refwd) makes x_{k+1} again from the kept intermediates of F_k^o, with
 * tmp(F_k^o), while x_k is live.
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
