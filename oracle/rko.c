/*
 * rko.c -- CPU oracle of the rk-Rotor dynamic program (Rockmate, App. C).
 *
 * TEST INFRASTRUCTURE ONLY: the slow, obviously correct reference that the HIP
 * path is compared with.  Plain C, one thread, 64-bit arithmetic, no blocking,
 * no fusion.  It shares nothing with the HIP library.  See rko.h for the
 * conventions (inclusive spans, budget beyond the span input, tie rule).
 */
#include "rko.h"

#include <stdlib.h>
#include <string.h>

int64_t rko_ncells(int32_t L) { return (int64_t)L * (L + 1) / 2; }

int64_t rko_cell(int32_t L, int32_t s, int32_t t)
{
    /* rows s' < s hold L - s' spans each */
    return (int64_t)s * L - (int64_t)s * (s - 1) / 2 + (t - s);
}

static int chain_ok(const rko_chain *c)
{
    if (!c || c->L < 1 || c->K < 1 || !c->x || !c->fn_time || !c->fn_tmp || !c->fwd || !c->bwd ||
        !c->mem || !c->tmp_fwd || !c->tmp_bwd)
        return 0;
    /* choice codes go up to L + K - 1 (L + 2K - 1 with the saving sweep) and fit int16 */
    if ((int64_t)c->L + (c->refwd ? 2 : 1) * (int64_t)c->K > 32767) return 0;
    return 1;
}

/* Opt(s, t, m) as stored; m must be in [0, M]. */
static int64_t get_opt(const rko_chain *c, const int32_t *opt, int64_t ncells, int32_t s, int32_t t,
                       int64_t m)
{
    return opt[m * ncells + rko_cell(c->L, s, t)];
}

/*
 * H(s, t, u) of the saving sweep (t > s), the rest of case 3 after F_{s-1}^o:
 * the sweep F_s^0 .. F_{i-1}^0 keeps x_i and drops everything behind it,
 * including its own input x_s (which the kept data of block s-1 can make
 * again), so every F_k^0 of it, k = s..i-1, needs its input x_k, its output
 * x_{k+1} and tmp(F_k^0) within u.  Then i..t runs with x_i held (u - x_i) and,
 * once x_s is back, s..i-1 with x_s held (u - x_s).  Code i; the smaller i wins
 * a tie.
 */
static void eval_h(const rko_chain *c, const int32_t *opt, int64_t ncells, int32_t s, int32_t t,
                   int64_t u, int64_t *best_cost, int32_t *best_code)
{
    int64_t best = RKO_INF;
    int32_t code = -1;
    int64_t sweep_time = 0, sweep_mem = 0;
    for (int32_t i = s + 1; i <= t; ++i) {
        int32_t k = i - 1;
        int64_t use = (int64_t)c->x[k] + c->x[k + 1] + c->fn_tmp[k];
        sweep_time += c->fn_time[k];
        if (use > sweep_mem) sweep_mem = use;
        if (sweep_mem > u) continue;
        int64_t right = get_opt(c, opt, ncells, i, t, u - c->x[i]);
        int64_t left = get_opt(c, opt, ncells, s, i - 1, u - c->x[s]);
        if (right >= RKO_INF || left >= RKO_INF) continue;
        int64_t v = sweep_time + right + left;
        if (v >= RKO_INF) continue;
        if (v < best) { best = v; code = i; }
    }
    *best_cost = best;
    *best_code = code;
}

/*
 * One cell of Eq. (all): Opt(s,t,m) = min(Opt_1, Opt_2) (and Opt_3 of the saving sweep).
 *
 * Case 2 (Eq. fn): block s is computed more than once.  The sweep runs
 * F_s^0, F_{s+1}^0, ..., F_{i-1}^0 keeping only x_i (x_{s+1}..x_{i-1} are
 * dropped right after their use); it costs the sum of r(F_k^0) and is valid
 * if every F_k^0 of the sweep fits in m: its input (not counted for k = s,
 * whose input is the span input), its output x_{k+1} and tmp(F_k^0).  Then
 * the subproblem i..t runs with x_i held (budget m - x_i), and afterwards
 * s..i-1 with the full budget.  Splits are i = s+1..t.
 *
 * Case 1 (Eq. fe): block s is computed once, with a saving option o.  F_s^o
 * leaves x_{s+1} and its intermediates, of total size xbar = x_{s+1} + mem;
 * it is valid if both F_s^o and B_s^o fit their temporary memory on top of
 * xbar; the rest of the span runs with m - xbar.  A single block (s = t) has
 * only this case, with an empty rest.
 *
 * Case 3 (the saving sweep, only with refwd; see rko.h): F_s^o as in case 1,
 * then H(s+1, t, m - mem) with its kept intermediates held throughout.
 *
 * Codes: split i -> i; option o -> L + o; saving sweep with option o ->
 * L + K + o.  The lexicographic minimum of (cost, code) is kept, which is what
 * Alg. 3 picks (case 2 before case 1 on equal cost; smaller i, then smaller o).
 */
static void eval_cell(const rko_chain *c, const int32_t *opt, const int32_t *hval, int64_t ncells,
                      int32_t s, int32_t t, int64_t m, int64_t *best_cost, int32_t *best_code)
{
    const int32_t L = c->L, K = c->K;
    int64_t best = RKO_INF;
    int32_t code = -1;

    if (t > s) {
        int64_t sweep_time = 0, sweep_mem = 0;
        for (int32_t i = s + 1; i <= t; ++i) {
            int32_t k = i - 1; /* F_k^0 is the last forward of this sweep */
            int64_t use = (k > s ? (int64_t)c->x[k] : 0) + c->x[k + 1] + c->fn_tmp[k];
            sweep_time += c->fn_time[k];
            if (use > sweep_mem) sweep_mem = use;
            if (sweep_mem > m) continue;
            int64_t right = get_opt(c, opt, ncells, i, t, m - c->x[i]);
            int64_t left = get_opt(c, opt, ncells, s, i - 1, m);
            if (right >= RKO_INF || left >= RKO_INF) continue;
            int64_t v = sweep_time + right + left;
            if (v >= RKO_INF) continue;
            if (v < best || (v == best && i < code)) { best = v; code = i; }
        }
    }
    for (int32_t o = 0; o < K; ++o) {
        int64_t xbar = (int64_t)c->x[s + 1] + c->mem[(int64_t)s * K + o];
        if (m < xbar + c->tmp_fwd[(int64_t)s * K + o]) continue;
        if (m < xbar + c->tmp_bwd[(int64_t)s * K + o]) continue;
        int64_t rest = 0;
        if (t > s) {
            rest = get_opt(c, opt, ncells, s + 1, t, m - xbar);
            if (rest >= RKO_INF) continue;
        }
        int64_t v = (int64_t)c->fwd[(int64_t)s * K + o] + c->bwd[(int64_t)s * K + o] + rest;
        if (v >= RKO_INF) continue;
        if (v < best || (v == best && L + o < code)) { best = v; code = L + o; }
    }
    /* Case 3 (the saving sweep, with refwd): F_s^o as in case 1 (same validity: F_s^o,
     * the recomputation of x_{s+1} and B_s^o all fit on top of xbar), its intermediates
     * held through H(s+1, t, .), which needs a split i >= s+2. */
    if (c->refwd && t >= s + 2) {
        for (int32_t o = 0; o < K; ++o) {
            int64_t mem = c->mem[(int64_t)s * K + o];
            int64_t xbar = (int64_t)c->x[s + 1] + mem;
            if (m < xbar + c->tmp_fwd[(int64_t)s * K + o]) continue;
            if (m < xbar + c->tmp_bwd[(int64_t)s * K + o]) continue;
            int64_t h = hval[(m - mem) * ncells + rko_cell(L, s + 1, t)];
            if (h >= RKO_INF) continue;
            int64_t v = (int64_t)c->fwd[(int64_t)s * K + o] + c->bwd[(int64_t)s * K + o] +
                        c->refwd[(int64_t)s * K + o] + h;
            if (v >= RKO_INF) continue;
            if (v < best || (v == best && L + K + o < code)) { best = v; code = L + K + o; }
        }
    }
    *best_cost = best;
    *best_code = code;
}

/* Alg. 2: for every budget m (outer loop), every span length, every start.  With the
 * saving sweep, H(s,t,m) is filled next to Opt(s,t,m): it reads Opt of shorter spans at
 * columns up to m, and Opt(s-1,t,.) reads H(s,t,.) at columns up to m. */
int rko_solve(const rko_chain *c, int32_t M, int32_t *opt, int16_t *arg, int32_t *hval, int16_t *harg,
              int32_t *answer)
{
    if (!chain_ok(c) || M < 0 || !opt || !arg || !answer) return RKO_E_INVAL;
    if (c->refwd && (!hval || !harg)) return RKO_E_INVAL;
    const int32_t L = c->L;
    const int64_t ncells = rko_ncells(L);
    for (int64_t m = 0; m <= M; ++m) {
        for (int32_t d = 0; d < L; ++d) {
            for (int32_t s = 0; s + d < L; ++s) {
                int64_t v;
                int32_t code;
                if (c->refwd) {
                    v = RKO_INF;
                    code = -1;
                    if (d > 0) eval_h(c, opt, ncells, s, s + d, m, &v, &code);
                    hval[m * ncells + rko_cell(L, s, s + d)] = (int32_t)v;
                    harg[m * ncells + rko_cell(L, s, s + d)] = (int16_t)code;
                }
                eval_cell(c, opt, hval, ncells, s, s + d, m, &v, &code);
                opt[m * ncells + rko_cell(L, s, s + d)] = (int32_t)v;
                arg[m * ncells + rko_cell(L, s, s + d)] = (int16_t)code;
            }
        }
    }
    if (M < c->x[0])
        *answer = RKO_INF;
    else
        *answer = opt[(int64_t)(M - c->x[0]) * ncells + rko_cell(L, 0, L - 1)];
    return RKO_OK;
}

/* ---- Alg. 3: rk-Rotor-Build ------------------------------------------------ */

typedef struct {
    rko_op *ops;
    int64_t cap, n, n_fwd;
    int bad;
} emitter;

static void emit(emitter *e, int32_t kind, int32_t block, int32_t option)
{
    if (kind == RKO_BWD && e->n_fwd < 0) e->n_fwd = e->n;
    if (e->ops && e->n < e->cap) {
        e->ops[e->n].kind = kind;
        e->ops[e->n].block = block;
        e->ops[e->n].option = option;
    }
    e->n++;
}

static void build(const rko_chain *c, const int16_t *arg, const int16_t *harg, int64_t ncells,
                  int32_t s, int32_t t, int64_t m, emitter *e)
{
    const int32_t L = c->L, K = c->K;
    int32_t code = arg[m * ncells + rko_cell(L, s, t)];
    if (code < 0) { e->bad = 1; return; }
    if (code >= L + K) {
        /* case 3 with option o: (F_s^o, F_{s+1}^0, ..., F_{i-1}^0, Build(i, t, u - x_i), REFWD_s^o,
         * Build(s+1, i-1, m - xbar), B_s^o) with u = m - mem and i the sweep's split at
         * H(s+1, t, u); each x_k (s < k < i) is dropped once F_k^0 has consumed it, x_i once
         * the subproblem i..t has finished with it. */
        int32_t o = code - L - K;
        int64_t mem = c->mem[(int64_t)s * K + o];
        int64_t u = m - mem;
        int32_t i = harg ? harg[u * ncells + rko_cell(L, s + 1, t)] : -1;
        if (!c->refwd || i < s + 2 || i > t) { e->bad = 1; return; }
        emit(e, RKO_FWD_SAVE, s, o);
        for (int32_t k = s + 1; k < i; ++k) {
            emit(e, RKO_FWD_NOSAVE, k, -1);
            emit(e, RKO_FREE_X, k, -1);
        }
        build(c, arg, harg, ncells, i, t, u - c->x[i], e);
        emit(e, RKO_FREE_X, i, -1);
        emit(e, RKO_REFWD, s, o);
        build(c, arg, harg, ncells, s + 1, i - 1, u - c->x[s + 1], e);
        emit(e, RKO_BWD, s, o);
    } else if (code >= L) {
        /* case 1 with option o: (F_s^o, Build(s+1, t, m - xbar), B_s^o) */
        int32_t o = code - L;
        int64_t xbar = (int64_t)c->x[s + 1] + c->mem[(int64_t)s * K + o];
        emit(e, RKO_FWD_SAVE, s, o);
        if (t > s) build(c, arg, harg, ncells, s + 1, t, m - xbar, e);
        emit(e, RKO_BWD, s, o);
    } else {
        /* case 2 with split i: (F_s^0, ..., F_{i-1}^0, Build(i, t, m - x_i), Build(s, i-1, m)),
         * dropping each x_k (s < k < i) once F_k^0 has consumed it and x_i once
         * the subproblem i..t has finished with it. */
        int32_t i = code;
        emit(e, RKO_FWD_NOSAVE, s, -1);
        for (int32_t k = s + 1; k < i; ++k) {
            emit(e, RKO_FWD_NOSAVE, k, -1);
            emit(e, RKO_FREE_X, k, -1);
        }
        build(c, arg, harg, ncells, i, t, m - c->x[i], e);
        emit(e, RKO_FREE_X, i, -1);
        build(c, arg, harg, ncells, s, i - 1, m, e);
    }
}

int rko_schedule(const rko_chain *c, int32_t M, const int16_t *arg, const int16_t *harg, rko_op *ops,
                 int64_t cap, int64_t *n_ops, int64_t *n_fwd)
{
    if (!chain_ok(c) || M < 0 || !arg || !n_ops || cap < 0) return RKO_E_INVAL;
    if (c->refwd && !harg) return RKO_E_INVAL;
    const int32_t L = c->L;
    const int64_t ncells = rko_ncells(L);
    if (M < c->x[0]) return RKO_E_INFEASIBLE;
    int64_t m = M - c->x[0];
    if (arg[m * ncells + rko_cell(L, 0, L - 1)] < 0) return RKO_E_INFEASIBLE;
    emitter e = {ops, cap, 0, -1, 0};
    build(c, arg, harg, ncells, 0, L - 1, m, &e);
    if (e.bad) return RKO_E_INVAL;
    *n_ops = e.n;
    if (n_fwd) *n_fwd = e.n_fwd;
    if (!ops || e.n > cap) return RKO_E_BUFSZ;
    return RKO_OK;
}

/* ---- replay ------------------------------------------------------------------ */

int rko_simulate(const rko_chain *c, const rko_op *ops, int64_t n, int64_t *time, int64_t *peak,
                 int64_t *bad)
{
    if (!chain_ok(c) || (n > 0 && !ops) || n < 0 || !time || !peak || !bad) return RKO_E_INVAL;
    const int32_t L = c->L, K = c->K;
    char *xlive = calloc((size_t)L + 1, 1);
    int32_t *hopt = malloc(sizeof(int32_t) * (size_t)L);
    char *gready = calloc((size_t)L + 1, 1);
    if (!xlive || !hopt || !gready) { free(xlive); free(hopt); free(gready); return RKO_E_INVAL; }
    for (int32_t k = 0; k < L; ++k) hopt[k] = -1;
    xlive[0] = 1;
    gready[L] = 1; /* the gradient of the chain output is given */
    int64_t used = c->x[0], pk = used, tm = 0;
    int64_t j;
    int err = 0;
    for (j = 0; j < n && !err; ++j) {
        int32_t kind = ops[j].kind, k = ops[j].block, o = ops[j].option;
        switch (kind) {
        case RKO_FWD_NOSAVE:
            if (k < 0 || k >= L || !xlive[k] || xlive[k + 1]) { err = 1; break; }
            if (used + c->x[k + 1] + c->fn_tmp[k] > pk) pk = used + c->x[k + 1] + c->fn_tmp[k];
            used += c->x[k + 1];
            xlive[k + 1] = 1;
            tm += c->fn_time[k];
            break;
        case RKO_FWD_SAVE: {
            if (k < 0 || k >= L || o < 0 || o >= K || !xlive[k] || xlive[k + 1] || hopt[k] >= 0) {
                err = 1;
                break;
            }
            int64_t add = (int64_t)c->x[k + 1] + c->mem[(int64_t)k * K + o];
            if (used + add + c->tmp_fwd[(int64_t)k * K + o] > pk)
                pk = used + add + c->tmp_fwd[(int64_t)k * K + o];
            used += add;
            xlive[k + 1] = 1;
            hopt[k] = o;
            tm += c->fwd[(int64_t)k * K + o];
            break;
        }
        case RKO_BWD:
            if (k < 0 || k >= L || o < 0 || o >= K || hopt[k] != o || !xlive[k] || !xlive[k + 1] ||
                !gready[k + 1] || gready[k]) {
                err = 1;
                break;
            }
            if (used + c->tmp_bwd[(int64_t)k * K + o] > pk) pk = used + c->tmp_bwd[(int64_t)k * K + o];
            used -= (int64_t)c->x[k + 1] + c->mem[(int64_t)k * K + o];
            xlive[k + 1] = 0;
            hopt[k] = -1;
            gready[k] = 1;
            tm += c->bwd[(int64_t)k * K + o];
            break;
        case RKO_REFWD:
            if (!c->refwd || k < 0 || k >= L || o < 0 || o >= K || hopt[k] != o || !xlive[k] || xlive[k + 1]) {
                err = 1;
                break;
            }
            if (used + c->x[k + 1] + c->tmp_fwd[(int64_t)k * K + o] > pk)
                pk = used + c->x[k + 1] + c->tmp_fwd[(int64_t)k * K + o];
            used += c->x[k + 1];
            xlive[k + 1] = 1;
            tm += c->refwd[(int64_t)k * K + o];
            break;
        case RKO_FREE_X:
            if (k < 1 || k > L || !xlive[k]) { err = 1; break; }
            used -= c->x[k];
            xlive[k] = 0;
            break;
        default:
            err = 1;
        }
    }
    int ok = !err;
    if (ok) {
        if (!gready[0] || !xlive[0]) ok = 0;
        for (int32_t k = 1; k <= L && ok; ++k)
            if (xlive[k]) ok = 0;
        for (int32_t k = 0; k < L && ok; ++k)
            if (hopt[k] >= 0) ok = 0;
        *bad = ok ? -1 : n;
    } else {
        *bad = j - 1;
    }
    *time = tm;
    *peak = pk;
    free(xlive);
    free(hopt);
    free(gready);
    return ok ? RKO_OK : RKO_E_REPLAY;
}

/* ---- feasibility threshold ----------------------------------------------------- */

static int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

int rko_min_feasible(const rko_chain *c, int64_t *out)
{
    if (!chain_ok(c) || !out) return RKO_E_INVAL;
    const int32_t L = c->L, K = c->K;
    /* hmin(s,t): smallest u at which H(s,t,u) is finite (saving sweep only) */
    int64_t *hmin = c->refwd ? malloc(sizeof(int64_t) * (size_t)rko_ncells(L)) : NULL;
    if (c->refwd && !hmin) return RKO_E_INVAL;
    for (int32_t d = 0; d < L; ++d) {
        for (int32_t s = 0; s + d < L; ++s) {
            int32_t t = s + d;
            int64_t best = INT64_MAX;
            if (hmin) {
                int64_t hb = INT64_MAX, sweep = 0;
                for (int32_t i = s + 1; i <= t; ++i) {
                    int32_t k = i - 1;
                    sweep = max64(sweep, (int64_t)c->x[k] + c->x[k + 1] + c->fn_tmp[k]);
                    int64_t need = max64(sweep, max64((int64_t)c->x[i] + out[rko_cell(L, i, t)],
                                                      (int64_t)c->x[s] + out[rko_cell(L, s, i - 1)]));
                    if (need < hb) hb = need;
                }
                hmin[rko_cell(L, s, t)] = hb;
                if (d >= 2)
                    for (int32_t o = 0; o < K; ++o) {
                        int64_t mem = c->mem[(int64_t)s * K + o];
                        int64_t xbar = (int64_t)c->x[s + 1] + mem;
                        int64_t h = hmin[rko_cell(L, s + 1, t)];
                        if (h == INT64_MAX) continue;
                        int64_t need = max64(max64(xbar + c->tmp_fwd[(int64_t)s * K + o],
                                                   xbar + c->tmp_bwd[(int64_t)s * K + o]),
                                             mem + h);
                        if (need < best) best = need;
                    }
            }
            for (int32_t o = 0; o < K; ++o) {
                int64_t xbar = (int64_t)c->x[s + 1] + c->mem[(int64_t)s * K + o];
                int64_t need = max64(xbar + c->tmp_fwd[(int64_t)s * K + o],
                                     xbar + c->tmp_bwd[(int64_t)s * K + o]);
                if (t > s) need = max64(need, xbar + out[rko_cell(L, s + 1, t)]);
                if (need < best) best = need;
            }
            int64_t sweep = 0;
            for (int32_t i = s + 1; i <= t; ++i) {
                int32_t k = i - 1;
                sweep = max64(sweep, (k > s ? (int64_t)c->x[k] : 0) + c->x[k + 1] + c->fn_tmp[k]);
                int64_t need = max64(sweep, max64((int64_t)c->x[i] + out[rko_cell(L, i, t)],
                                                  out[rko_cell(L, s, i - 1)]));
                if (need < best) best = need;
            }
            out[rko_cell(L, s, t)] = best;
        }
    }
    free(hmin);
    return RKO_OK;
}
