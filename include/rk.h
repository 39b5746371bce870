/*
 * rk.h -- C ABI of librkrotor, the rk-Rotor solver of Rockmate (arXiv 2307.01236)
 * on AMD Instinct MI355X (gfx950).
 *
 * The library computes rk-Rotor's dynamic program (App. C, Eqs. fe, fn and
 * all; Alg. 2) on the GPU and turns its optimum into a compute/forget
 * schedule (Alg. 3).  It plays the role of the line of Rockmate's Alg. 1 that
 * produces Sequence = rk-Rotor(sols, M_GPU): the per-block option sets come in
 * through rk_chain_create, the budget through rk_solve, and the schedule
 * comes out of rk_extract_schedule.
 *
 * Model (App. C notation, 0-based):
 *   - blocks 0..L-1; activation x_i is the input of block i, x_L the output;
 *   - F_i^0 is the forward that keeps nothing: time r(F_i^0) = fn_time[i],
 *     temporary memory tmp(F_i^0) = fn_tmp[i];
 *   - each block has K saving options o = 0..K-1: forward F_i^o (time
 *     fwd[i*K+o], temporary tmp_fwd[i*K+o]) which keeps mem[i*K+o] slots of
 *     intermediates until the backward B_i^o (time bwd[i*K+o], temporary
 *     tmp_bwd[i*K+o]).  The paper's xbar_i^o is x_{i+1} + mem[i*K+o];
 *   - Opt(s,t,m) is the best time for blocks s..t (inclusive) when x_s stays
 *     live and m slots are available beyond it; the answer for a budget M is
 *     Opt(0, L-1, M - x_0);
 *   - sizes, budgets and times are non-negative integers (memory "slots" and
 *     time units of the caller's choosing); all arithmetic is exact.
 *
 * Ties: when several choices reach the optimum the one recorded is the
 * lexicographic minimum of (cost, code) with code = i for the case-2 split
 * that keeps x_i and code = L + o for the case-1 option o (Alg. 3 tests case 2
 * before case 1; smaller i, then smaller o).  This makes every table and
 * schedule unique.
 *
 * Threading: a chain is not thread-safe; distinct chains are independent.
 * Device: the library works on the HIP device current at the first solve of
 * a chain and keeps using it for that chain.
 * Errors: every call returns an RK_* code; nothing is thrown across the ABI.
 */
#ifndef RK_H
#define RK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RK_INF INT32_MAX                  /* "no valid schedule" (Eq. all: +infinity)    */
#define RK_TIME_LIMIT ((int32_t)((1 << 30) - 2)) /* largest admissible schedule-time bound */
#define RK_MAX_L 2000                     /* longest chain                                */
#define RK_MAX_M ((int32_t)((1 << 26) - 2))       /* largest budget                       */

enum { RK_FWD_NOSAVE = 0, RK_FWD_SAVE = 1, RK_BWD = 2, RK_FREE_X = 3, RK_REFWD = 4 };

enum {
    RK_OK = 0,
    RK_E_INVAL = -1,       /* bad argument (NULL, negative, out of range)                    */
    RK_E_OVERFLOW = -2,    /* schedule times could exceed RK_TIME_LIMIT                       */
    RK_E_NOMEM = -3,       /* device or host allocation failed, or workspace too small        */
    RK_E_DEVICE = -4,      /* a HIP call failed (no device, launch error, ...)                */
    RK_E_NOT_SOLVED = -5,  /* no completed solve to read from                                 */
    RK_E_INFEASIBLE = -6,  /* the budget admits no schedule                                   */
    RK_E_BUFSZ = -7,       /* caller buffer too small; the needed size was returned           */
    RK_E_INTERNAL = -8     /* a consistency check inside the library failed                    */
};

/* One schedule step.  kind: RK_FWD_NOSAVE (F_block^0), RK_FWD_SAVE (F_block^option),
 * RK_BWD (B_block^option), RK_FREE_X (drop activation x_block), RK_REFWD (make
 * x_{block+1} again from the intermediates F_block^option kept; the saving sweep only).
 * option is -1 for RK_FWD_NOSAVE and RK_FREE_X. */
typedef struct { int32_t kind, block, option; } rk_op;

typedef struct rk_chain rk_chain;

/*
 * Create a chain from its per-block option sets (Alg. 1: the sols of every
 * block; App. C notation).  All arrays are host memory and are deep-copied,
 * so the caller may free them on return.  Layouts: x [L+1]; fn_time, fn_tmp
 * [L]; fwd, bwd, mem, tmp_fwd, tmp_bwd [L*K] row-major (option fastest).
 * Checks: 1 <= L <= RK_MAX_L, K >= 1, L + K < 32768, every entry >= 0, and the
 * bound on any schedule's time, L * sum_i max(fn_time_i, max_o fwd_i^o) +
 * sum_i max_o bwd_i^o, must not exceed RK_TIME_LIMIT (else RK_E_OVERFLOW).
 * Does not touch the GPU.  On success *out owns a new chain.
 */
int rk_chain_create(int32_t L, int32_t K, const int32_t *x, const int32_t *fn_time,
                    const int32_t *fn_tmp, const int32_t *fwd, const int32_t *bwd,
                    const int32_t *mem, const int32_t *tmp_fwd, const int32_t *tmp_bwd,
                    rk_chain **out);

/*
 * The saving sweep: this library's reading of the sub-optimality remark (ii) of Sec. 3.4
 * (a forward that runs several times may keep intermediate data on its first pass and use
 * it to make its output faster on later passes).  It adds a third case to Eq. all for a
 * span (s,t) with t >= s+2 and a saving option o of block s: F_s^o keeps its intermediates,
 * the no-save forwards F_{s+1}^0 .. F_{i-1}^0 run to x_i dropping everything behind them
 * (x_{s+1} included), blocks i..t are solved with x_i held, x_i is dropped, x_{s+1} is made
 * again from the kept data (an RK_REFWD step of time refwd[s*K+o] and temporary memory
 * tmp_fwd[s*K+o]), blocks s+1..i-1 are solved, and B_s^o ends the span:
 *   Opt_3(s,t,m) = min_o r(F_s^o) + r(B_s^o) + refwd_s^o + H(s+1, t, m - mem_s^o),
 *   H(s',t,u)   = min_{i=s'+1..t} sum_{k=s'}^{i-1} r(F_k^0) + Opt(i,t,u - x_i) + Opt(s',i-1,u - x_s'),
 * valid where case 1 with o is, and where every F_k^0 of the sweep fits u with its input,
 * its output and tmp(F_k^0).  The recorded choice of case 3 has code L + K + o (after case
 * 2's codes i and case 1's codes L + o).
 * refwd: host [L*K] re-forward times (deep-copied), or NULL to switch the case off (the
 * default).  Takes effect at the next solve; the workspace of a solve with the case on
 * holds twice the tables.  RK_E_INVAL for a negative time or L + 2K >= 32768,
 * RK_E_OVERFLOW when L * sum_i max(r(F_i^0), max_o r(F_i^o), max_o refwd_i^o) +
 * sum_i max_o r(B_i^o) exceeds RK_TIME_LIMIT; the chain is unchanged then.
 */
int rk_chain_set_saving_sweep(rk_chain *c, const int32_t *refwd);

/* Release the chain, its device copies and any table it allocated.  NULL is a no-op. */
void rk_chain_destroy(rk_chain *c);

/* Bytes of device workspace a solve of this chain at budget M needs (the
 * Opt table over every span and every m <= M that Alg. 2 fills, and its companions).  RK_E_INVAL for M outside [0, RK_MAX_M];
 * RK_E_NOMEM when 18L + 64 table rows would span 2 GiB or more (the kernels
 * address operand blocks with 32-bit offsets; at L = 384 this allows budgets up
 * to about 77 000) or the tables exceed 2^40 int32. */
int rk_workspace_bytes(const rk_chain *c, int32_t M, size_t *bytes);

/*
 * Fill Opt(s,t,m) for every span and every m in [0, M] (Alg. 2) in a table
 * the chain allocates (and reuses across solves), then return the answer
 * Opt(0, L-1, M - x_0) in *opt_out, or RK_INF when the budget admits no
 * schedule (including M < x_0).  Synchronous; runs on a stream the chain owns.
 * RK_E_NOMEM if the table cannot be allocated, RK_E_DEVICE on a HIP error.
 */
int rk_solve(rk_chain *c, int32_t M, int32_t *opt_out);

/*
 * Same fill, asynchronous, in caller memory: d_workspace is device memory of
 * at least rk_workspace_bytes(c, M) bytes (for instance a torch tensor) and
 * stream a hipStream_t (NULL: a stream the chain owns).  Returns once the work
 * is queued.  The fill's kernel sequence is captured into a HIP graph on first
 * use and replayed while M, the workspace, the stream and the profiling switch
 * stay the same.  The workspace must stay allocated and untouched until the
 * chain is destroyed or solved again; the chain reads results from it.  Call
 * rk_result to wait and read the answer.
 *
 * On a stream the caller is capturing into a HIP graph, the kernels are launched
 * directly and become part of the caller's graph; nothing is allocated, uploaded or
 * waited on.  That needs a chain solved once before (outside the capture, with the
 * same option-pruning setting), a caller workspace, and profiling off, else
 * RK_E_INVAL.  Each replay of the caller's graph refills the table.  The library
 * cannot wait for the caller's replays: the caller synchronizes the stream it replays
 * on before rk_result, rk_read_row, rk_tradeoff_curve or rk_extract_schedule, which then
 * read the last replay's results without waiting; rk_last_fill_ms returns RK_E_INVAL
 * for such a fill.  The same holds for rk_solve_noalloc on a stream under capture.
 */
int rk_solve_async(rk_chain *c, int32_t M, void *d_workspace, size_t ws_bytes, void *stream);

/*
 * For callers that cannot allocate (code under HIP graph capture that may not call
 * hipMalloc, tight serving loops, harnesses that forbid allocation): the fill of
 * rk_solve_async, with its tables in a static device array of RK_NOALLOC_MAX_BYTES that
 * the library holds on every device it runs on (until the process ends), and with its
 * kernels launched one by one on `stream` (NULL: a stream the chain owns).  This call
 * allocates nothing: no hipMalloc, hipFree, graph or event creation.  Asynchronous like
 * rk_solve_async; rk_result, rk_read_row, rk_tradeoff_curve and rk_extract_schedule
 * then read that array.
 *   - The chain must have been solved once before on this device (rk_solve or
 *     rk_solve_async, which upload its derived arrays), with the same option-pruning
 *     setting, and profiling must be off; else RK_E_INVAL.
 *   - RK_E_NOMEM when rk_workspace_bytes(c, M) exceeds RK_NOALLOC_MAX_BYTES (about
 *     L = 64 blocks at M = 2500, or L = 128 at M = 575, with activations of at most
 *     64 slots).
 *   - Every call on a device shares that device's array and overwrites what the previous
 *     call left there: reads of an earlier call's results are valid only until the next
 *     rk_solve_noalloc on the same device, and calls that overlap on one device (other
 *     streams, other threads, other chains) race.
 */
#define RK_NOALLOC_MAX_BYTES ((size_t)64 << 20)
int rk_solve_noalloc(rk_chain *c, int32_t M, void *stream);

/* Wait for the last solve of the chain and return its answer (as rk_solve). */
int rk_result(rk_chain *c, int32_t *opt_out);

/*
 * Alg. 3 (rk-Rotor-Build) for the last solve's budget: the schedule as a list
 * of steps, with every forget of an activation made explicit.  The choice at
 * each visited (s,t,m) is recomputed on the GPU from the finished Opt table
 * (the lexicographic (cost, code) minimum).  Two-call: with ops == NULL or
 * cap smaller than the schedule, *n_ops receives its length and RK_E_BUFSZ is
 * returned.  *n_fwd (may be NULL) receives the index of the first backward,
 * i.e. the split between Sequence.fwd and Sequence.bwd.  RK_E_NOT_SOLVED
 * before a solve, RK_E_INFEASIBLE when the answer is RK_INF.
 */
int rk_extract_schedule(rk_chain *c, rk_op *ops, int64_t cap, int64_t *n_ops, int64_t *n_fwd);

/*
 * Copy row (s,t) of the last solve: opt_row[m] = Opt(s,t,m), the optimal time of
 * the span s..t within budget m (App. C, Eq. all; RK_INF where
 * infeasible) and arg_row[m] = the recorded choice code (-1 where infeasible),
 * for m = 0..M; each buffer holds M+1 entries and either may be NULL.
 * RK_E_INVAL unless 0 <= s <= t < L.
 */
int rk_read_row(rk_chain *c, int32_t s, int32_t t, int32_t *opt_row, int16_t *arg_row);

/*
 * The memory/time trade-off of the last solve, the curve of the paper's
 * comparison with Rotor (Sec. 4, overhead against peak memory): times[b] is the
 * best schedule time within a total budget of b slots, Opt(0, L-1, b - x_0), or
 * RK_INF when b < x_0 or no schedule fits, for b = 0 .. n-1.  One fill at budget
 * M answers every smaller budget (Alg. 2 fills all m <= M), so n may be at most
 * M + 1 of the last solve.  times is host memory the caller owns.  RK_E_INVAL
 * for n outside [0, M + 1] or NULL times with n > 0; RK_E_NOT_SOLVED before a solve.
 */
int rk_tradeoff_curve(rk_chain *c, int32_t *times, int64_t n);

/*
 * Device time of the last solve's table fill, in milliseconds (HIP events
 * around the fill on the solve's stream), and the number of kernels launched.
 */
int rk_last_fill_ms(rk_chain *c, float *ms, int32_t *launches);

/*
 * Kernel-level timing (for benchmarks; mode 0, off, by default).  In mode 1 or 2 the
 * fill launches its kernels one by one instead of replaying a graph, and the runtime
 * records a pair of HIP events with every dispatch, at the kernel's start and end
 * (hipExtLaunchKernelGGL), so a launch's time is the kernel's own.  Mode 2 also runs
 * the counting variants of the fill kernels, which add up on the device the candidates
 * that only the kernels know to skip (slower: take timings from a mode-1 solve).
 * rk_fill_kernel_stats then reports, for kernel kind `kind` (0 <= kind < *n_kinds), its
 * name as a profiler shows it, the number of its launches in the last solve, their
 * summed device time in milliseconds, and three counts of the last profiled solve:
 *   - relaxations: candidate evaluations of the recurrence the launches cover (valid
 *     (s,t,m,choice) combinations, with k_run option slots per block; see
 *     rk_chain_options);
 *   - evaluated: those the kernels actually evaluate.  Past the budget msa(s,t) from
 *     which storing every activation of span (s,t) fits, Opt(s,t,m) is known in closed
 *     form (the sum of its blocks' cheapest r(F)+r(B), App. C: Opt can never be lower,
 *     and case 1 with those options reaches it); tiles whose cells all lie there skip.
 *     After a mode-2 solve, candidates skipped by a lower bound are left out as well:
 *     every case-2 candidate of span (s,t) at split i costs at least lb(s,t) + P(s,i),
 *     lb(s,t) being that closed form and P(s,i) the time of the plain forward sweep from
 *     block s to block i-1 (the band products count what they relax; mids and finalizes,
 *     what they skip);
 *   - bytes: compulsory table traffic of what runs: every table row a running tile
 *     reads, counted once over its budget columns, plus every row written (and read
 *     back where a fold into a stored partial happens).  After a mode-2 solve, only the
 *     rows that the candidates left after the lower-bound skips read.  (A mid tile
 *     tests its bound against partials that other tiles of its launch may be lowering at
 *     that moment, so its counts can differ slightly from solve to solve.)
 * Any output pointer may be NULL.  Waits for the last solve; timings and the last two
 * counts need profiling to have been on during it.  RK_E_INVAL for a kind or mode out
 * of range.
 */
int rk_set_profiling(rk_chain *c, int32_t mode);
int rk_fill_kernel_stats(rk_chain *c, int32_t kind, int32_t *n_kinds, const char **name,
                         int32_t *launches, float *total_ms, int64_t *relaxations, int64_t *evaluated,
                         int64_t *bytes);

/*
 * Options the solver evaluates (Sec. 3, Phase 2: the paper's option search returns many
 * repeated solutions for the budget grid, and rk-Rotor needs only the distinct ones).
 * Before the fill, option o of block s is dropped when an earlier option o' < o of the
 * same block is at least as good in everything Eq. fe reads: r(F)+r(B), xbar and the
 * memory the pair needs.  Then o' is a candidate wherever o is, never costs more (Opt is
 * non-increasing in m) and wins ties by its smaller code, so every Opt value, every
 * recorded choice and every schedule stay exactly as without the test; only the work
 * shrinks.  Repeated options are the special case of equality.  Options and recorded
 * choices always use the caller's option indices.
 *
 * rk_set_option_pruning: on (non-zero, the default) or off (every option evaluated, for
 * measurement); takes effect at the next solve.
 * rk_chain_options: kept[s*K + o] (host, [L*K], may be NULL) = 1 when option o of block
 * s is evaluated under the current setting; *k_run (may be NULL) = option slots per block
 * the kernels evaluate, the largest kept count (blocks with fewer are padded with slots
 * that never win).  Does not touch the GPU.
 */
int rk_set_option_pruning(rk_chain *c, int32_t enable);
int rk_chain_options(const rk_chain *c, int32_t *kept, int32_t *k_run);

/* Short English description of an RK_* code. */
const char *rk_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif /* RK_H */
