"""Randomized full-table parity of the HIP path against the oracle, longer than the test
suite runs (needs an MI355X; not collected by pytest).

    python tests/fuzz_parity.py N SEED [small|big|big4]

small (default): chains of 1-89 blocks with 1-39 options (sizes and times may be zero, a
quarter with identical blocks, a few time values only for ties), budgets from 0 to a bit
above storing everything; every fourth chain is short with a budget near 1.6e6 / L
columns, on either side of the width-4 mid level's threshold.  big: 90-199 blocks,
budgets below 350 (several bands, every mid width but 4).  big4: 64-109 blocks with
tables past the threshold (several bands and the width-4 level).  Option pruning
alternates.  Every chain's Opt table, choice table, answer and schedule must be
identical.  Exit status 1 if any differs.
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2307_01236_amd import rk  # noqa: E402
from paper_2307_01236_amd.chaingen import make_random_chain  # noqa: E402


def draw(it: int, seed: int, mode: str):
    rng = np.random.default_rng(seed)
    if mode == "big4":
        L = int(rng.integers(64, 110))
        K = int(rng.integers(1, 4))
        M = int(rng.integers(1_600_000 // L, 1_600_000 // L + 3000))
        ch = make_random_chain(seed, L, K, M=M, xmax=int(rng.integers(1, 300)), amax=int(rng.integers(1, 1500)),
                               tmax=int(rng.integers(0, 300)), tmin=0, allow_zero=bool(rng.integers(0, 2)),
                               small_times=bool(rng.integers(0, 2)))
    elif mode == "big":
        L = int(rng.integers(90, 200))
        K = int(rng.integers(1, 20))
        ch = make_random_chain(seed, L, K, xmax=int(rng.integers(1, 12)), amax=int(rng.integers(1, 20)),
                               tmax=int(rng.integers(0, 12)), tmin=0, allow_zero=bool(rng.integers(0, 2)),
                               small_times=bool(rng.integers(0, 2)))
        M = int(rng.integers(0, 350))
    elif it % 4 == 3:
        L = int(rng.integers(2, 26))
        K = int(rng.integers(1, 6))
        M = int(rng.integers(1_600_000 // L - 2000, 1_600_000 // L + 5000))
        ch = make_random_chain(seed, L, K, M=M, xmax=int(rng.integers(1, 200)), amax=int(rng.integers(1, 3000)),
                               tmax=int(rng.integers(0, 500)), tmin=0, allow_zero=bool(rng.integers(0, 2)))
    else:
        L = int(rng.integers(1, 90))
        K = int(rng.integers(1, 40))
        ch = make_random_chain(seed, L, K, xmax=int(rng.integers(1, 40)), amax=int(rng.integers(1, 90)),
                               tmax=int(rng.integers(0, 40)), tmin=0, allow_zero=bool(rng.integers(0, 2)),
                               small_times=bool(rng.integers(0, 2)), uniform=bool(rng.integers(0, 4) == 0))
        M = int(rng.integers(0, ch.M + 50))
    return ch, M


def same(ch, M, prune: bool) -> bool:
    sol = oracle.solve(ch, M)
    s = rk.Solver(ch)
    try:
        s.set_option_pruning(prune)
        ans = s.solve(M)
        g_opt, g_arg = s.rows()
        o_opt, o_arg = sol.rows()
        ok = ans == sol.answer and np.array_equal(g_opt, o_opt) and np.array_equal(g_arg, o_arg)
        exp = oracle.schedule(sol, M)
        if exp is not None:
            ops, nf = s.schedule()
            ok = ok and np.array_equal(ops, exp[0]) and nf == exp[1]
        return ok
    finally:
        s.close()


def main():
    n, seed0 = int(sys.argv[1]), int(sys.argv[2])
    mode = sys.argv[3] if len(sys.argv) > 3 else "small"
    t0, bad = time.time(), 0
    for it in range(n):
        ch, M = draw(it, seed0 + it, mode)
        if not same(ch, M, prune=bool(it % 2)):
            bad += 1
            print(f"MISMATCH chain {it} (seed {seed0 + it}): L={ch.L} K={ch.K} M={M}", flush=True)
        if it % 5 == 0:
            print(f"{it + 1} of {n} chains, {bad} differ, {time.time() - t0:.0f} s", flush=True)
    print(f"{n} chains, {bad} differ", flush=True)
    sys.exit(1 if bad else 0)


if __name__ == "__main__":
    main()
