"""Randomized full-table parity of the HIP path against the oracle, on fixed seeds.

Three kinds of chains, every one compared in full (Opt table, choice table, answer,
schedule), with option pruning alternating:
- small: 1-89 blocks, 1-39 options, sizes and times that may be zero, a quarter with
  identical blocks, a few time values only (ties), budgets from 0 to a bit above storing
  everything; every fourth chain is short with a budget near 1.6e6 / L columns (thousands
  of column chunks, large left pads);
- big: 90-199 blocks with budgets below 350 (several bands, both mid widths);
- big4: 64-109 blocks with tables of at least 1.6e6 blocks x budget columns (several bands,
  both mid widths, a few hundred column chunks).
"""
import numpy as np
import pytest

import oracle
from paper_2307_01236_amd import rk
from paper_2307_01236_amd.chaingen import make_random_chain

pytestmark = pytest.mark.gpu


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


def check_same(ch, M, prune: bool, where: str) -> None:
    print(f"  {where}: L={ch.L} K={ch.K} M={M} pruning={prune}", flush=True)
    sol = oracle.solve(ch, M)
    s = rk.Solver(ch)
    try:
        s.set_option_pruning(prune)
        ans = s.solve(M)
        g_opt, g_arg = s.rows()
        o_opt, o_arg = sol.rows()
        assert ans == sol.answer, (where, ans, sol.answer)
        assert np.array_equal(g_opt, o_opt), (where, "Opt", np.argwhere(g_opt != o_opt)[:3].tolist())
        assert np.array_equal(g_arg, o_arg), (where, "choice", np.argwhere(g_arg != o_arg)[:3].tolist())
        exp = oracle.schedule(sol, M)
        if exp is None:
            with pytest.raises(rk.RKError):
                s.schedule()
        else:
            ops, nf = s.schedule()
            assert np.array_equal(ops, exp[0]) and nf == exp[1], (where, "schedule")
    finally:
        s.close()


@pytest.mark.parametrize("group", range(4))
def test_fuzz_small_chains(group):
    """40 chains in four groups of ten (seeds 310000 + it)."""
    for it in range(10 * group, 10 * group + 10):
        ch, M = draw(it, 310000 + it, "small")
        check_same(ch, M, prune=bool(it % 2), where=f"small chain {it} (seed {310000 + it})")


@pytest.mark.parametrize("it", range(2))
def test_fuzz_big_chains(it):
    ch, M = draw(it, 320000 + it, "big")
    check_same(ch, M, prune=bool(it % 2), where=f"big chain {it} (seed {320000 + it})")


@pytest.mark.parametrize("it", range(4))
def test_fuzz_width4_chains(it):
    ch, M = draw(it, 330000 + it, "big4")
    check_same(ch, M, prune=bool(it % 2), where=f"big4 chain {it} (seed {330000 + it})")
