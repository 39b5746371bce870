/* Runs the CPU oracle (oracle/rko.c) on chains read from a file, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer.  File: per chain, int32 L, K, M,
 * has_refwd, then x[L+1], fn_time[L], fn_tmp[L], fwd, bwd, mem, tmp_fwd, tmp_bwd [L*K]
 * and refwd [L*K] when has_refwd.  Prints per chain: answer, sum of finite Opt values,
 * sum of choice codes, schedule length and the replay's time and peak, the sum of the
 * budget-free feasibility thresholds. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "rko.h"

static int32_t *take(FILE *f, size_t n)
{
    int32_t *p = malloc(sizeof(int32_t) * (n ? n : 1));
    if (!p || fread(p, sizeof(int32_t), n, f) != n) exit(3);
    return p;
}

int main(int argc, char **argv)
{
    if (argc != 2) return 2;
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int32_t hdr[4];
    while (fread(hdr, sizeof(int32_t), 4, f) == 4) {
        const int32_t L = hdr[0], K = hdr[1], M = hdr[2];
        const size_t nk = (size_t)L * K;
        rko_chain c;
        c.L = L;
        c.K = K;
        c.x = take(f, (size_t)L + 1);
        c.fn_time = take(f, (size_t)L);
        c.fn_tmp = take(f, (size_t)L);
        c.fwd = take(f, nk);
        c.bwd = take(f, nk);
        c.mem = take(f, nk);
        c.tmp_fwd = take(f, nk);
        c.tmp_bwd = take(f, nk);
        c.refwd = hdr[3] ? take(f, nk) : NULL;
        const int64_t n = rko_ncells(L), cells = n * ((int64_t)M + 1);
        int32_t *opt = malloc(sizeof(int32_t) * cells), *hval = malloc(sizeof(int32_t) * cells);
        int16_t *arg = malloc(sizeof(int16_t) * cells), *harg = malloc(sizeof(int16_t) * cells);
        int64_t *mf = malloc(sizeof(int64_t) * n);
        int32_t ans = 0;
        if (!opt || !hval || !arg || !harg || !mf) return 4;
        if (rko_solve(&c, M, opt, arg, hval, harg, &ans) != RKO_OK) return 5;
        int64_t osum = 0, asum = 0, mfs = 0;
        for (int64_t j = 0; j < cells; ++j) {
            if (opt[j] != RKO_INF) osum += opt[j];
            asum += arg[j];
        }
        if (rko_min_feasible(&c, mf) != RKO_OK) return 6;
        for (int64_t j = 0; j < n; ++j) mfs += mf[j] > 1000000000 ? 0 : mf[j];
        int64_t nops = 0, nfwd = 0, tm = -1, pk = -1, bad = 0;
        if (ans != RKO_INF) {
            if (rko_schedule(&c, M, arg, harg, NULL, 0, &nops, &nfwd) != RKO_E_BUFSZ) return 7;
            rko_op *ops = malloc(sizeof(rko_op) * (size_t)nops);
            if (!ops || rko_schedule(&c, M, arg, harg, ops, nops, &nops, &nfwd) != RKO_OK) return 8;
            if (rko_simulate(&c, ops, nops, &tm, &pk, &bad) != RKO_OK) return 9;
            free(ops);
        }
        printf("%d %lld %lld %lld %lld %lld %lld\n", ans, (long long)osum, (long long)asum, (long long)nops,
               (long long)tm, (long long)pk, (long long)mfs);
        free((void *)c.x); free((void *)c.fn_time); free((void *)c.fn_tmp); free((void *)c.fwd);
        free((void *)c.bwd); free((void *)c.mem); free((void *)c.tmp_fwd); free((void *)c.tmp_bwd);
        free((void *)c.refwd);
        free(opt); free(hval); free(arg); free(harg); free(mf);
    }
    fclose(f);
    return 0;
}
