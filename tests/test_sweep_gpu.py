"""The saving sweep (case 3, rk_chain_set_saving_sweep) on the MI355X against the oracle:
whole Opt and choice tables (case 3's codes L + K + o included), answers and schedules
(with their re-forward steps), on chains that exercise every level of the fill: the
diagonal finalize, mid products of every width and the band products, option pruning,
and switching the case on and off on one chain handle."""
import numpy as np
import pytest

import oracle
from paper_2307_01236_amd import rk
from paper_2307_01236_amd.chaingen import (make_config_chain, make_grid_chain, make_random_chain, store_all_bound,
                                            with_refwd)
from test_parity_gpu import check_same_schedule, full_parity, say

pytestmark = pytest.mark.gpu
INF = rk.RK_INF


@pytest.mark.parametrize("cfg", [0, 1])
def test_configs_with_sweep_full_tables(cfg):
    ch = with_refwd(make_config_chain(cfg), 11 + cfg, 0.0, 0.5)
    full_parity(ch)
    # a tight budget, where the re-forward pays
    mf = oracle.min_feasible(ch)[oracle.cell_index(ch.L)[0, ch.L - 1]]
    full_parity(ch, int(mf + ch.x[0] + 3))


def small_sweep_chains():
    out = []
    rng = np.random.default_rng(4040)
    for seed in range(10):
        L = int(rng.integers(1, 30))
        K = int(rng.integers(1, 9))
        ch = make_random_chain(4100 + seed, L, K, allow_zero=seed % 3 == 0, small_times=seed % 2 == 0,
                               uniform=seed % 4 == 3, xmax=int(rng.integers(1, 12)), amax=int(rng.integers(0, 20)),
                               tmax=int(rng.integers(0, 8)), tmin=0)
        ch = with_refwd(ch, seed, 0.0, 1.0 if seed % 5 else 0.0)
        hi = store_all_bound(ch)
        out.append((ch, int(rng.choice([0, 1, hi // 3, hi // 2, hi, 257]))))
    return out


@pytest.mark.parametrize("idx", range(10))
def test_small_chains_with_sweep(idx):
    ch, M = small_sweep_chains()[idx]
    full_parity(ch, M, prune=idx % 2 == 0)


@pytest.mark.parametrize("seed", [0, 1])
def test_multi_band_chains_with_sweep(seed):
    """90-110 blocks: band products at 32, 64 (and 96), every mid width but 4."""
    rng = np.random.default_rng(5150 + seed)
    L = int(rng.integers(90, 111))
    ch = make_random_chain(5150 + seed, L, int(rng.integers(2, 6)), xmax=8, amax=20, tmax=6, tmin=0)
    ch = with_refwd(ch, seed, 0.0, 0.7)
    full_parity(ch, min(store_all_bound(ch) // 3, 400), prune=seed == 0)


def test_large_table_with_sweep():
    """64 blocks x 25 001 budget columns: the mid products of widths 16 and 8 run for H too,
    and the finalize covers the splits whose longer operand spans the last 8 spans."""
    ch = make_random_chain(6464, 64, 3, xmax=50, amax=400, tmax=100, tmin=0)
    full_parity(with_refwd(ch, 3, 0.0, 0.5), 25000)


def test_wide_budget_with_sweep():
    """200 001 budget columns on 12 blocks with large sizes: H's left pad and shifts far
    beyond the finalize's staged halo."""
    ch = make_random_chain(777, 12, 3, xmax=2000, amax=9000, tmax=3000, tmin=0)
    full_parity(with_refwd(ch, 3, 0.0, 0.5), 200000)


def test_grid_options_with_sweep_pruned_and_unpruned():
    ch = with_refwd(make_grid_chain(8, 12, 6, 6), 5, 0.0, 0.4)
    for prune in (True, False):
        full_parity(ch, prune=prune)


def test_sweep_switched_on_and_off():
    base = make_config_chain(1)
    sw = with_refwd(base, 21, 0.0, 0.3)
    M = int(oracle.min_feasible(base)[oracle.cell_index(base.L)[0, base.L - 1]] + base.x[0] + 5)
    s = rk.Solver(base)
    try:
        for chain in (base, sw, base, sw):
            s.set_saving_sweep(chain.refwd)
            sol = oracle.solve(chain, M)
            assert s.solve(M) == sol.answer
            g_opt, g_arg = s.rows()
            o_opt, o_arg = sol.rows()
            assert np.array_equal(g_opt, o_opt) and np.array_equal(g_arg, o_arg)
            check_same_schedule(s, sol, chain, M)
    finally:
        s.close()


def test_sweep_lowers_answers_and_schedules_replay():
    """Where the re-forward pays, the answer drops below the unwidened one and the schedule
    replays in the oracle's simulator with re-forward steps, at its optimum's time."""
    base = make_config_chain(1)
    sw = with_refwd(base, 31, 0.0, 0.2)
    mf = int(oracle.min_feasible(sw)[oracle.cell_index(sw.L)[0, sw.L - 1]] + sw.x[0])
    found = False
    for M in range(mf, mf + 40, 4):
        s, t = rk.Solver(sw), rk.Solver(base)
        try:
            a, b = s.solve(M), t.solve(M)
            assert a <= b
            ops, _ = s.schedule()
            ok, tm, pk, _ = oracle.simulate(sw, ops)
            assert ok and tm == a and pk <= M
            found |= a < b and (ops[:, 0] == rk.RK_REFWD).any()
        finally:
            s.close()
            t.close()
    assert found
