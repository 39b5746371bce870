"""Option pruning before the fill (no GPU).

The library drops, per block, every option that an earlier option of the same block
matches or beats in all Eq. fe reads (r(F)+r(B), xbar, the memory the pair needs), and
claims that this leaves every Opt value and every recorded choice unchanged.  The first
test re-derives the kept set independently; the second checks the claim with the oracle
on chains rebuilt from the kept options only.
"""
import numpy as np

import oracle
from paper_2307_01236_amd import rk
from paper_2307_01236_amd.chaingen import Chain, make_config_chain, make_grid_chain, make_random_chain


def _handle(ch):
    return rk.rk_chain_create(ch.L, ch.K, *ch.arrays())


def reference_kept(ch):
    """Kept flags by the rule, written directly from the chain's arrays."""
    xb = ch.x[1:, None].astype(np.int64) + ch.mem
    need = xb + np.maximum(ch.tmp_fwd, ch.tmp_bwd)
    c1 = ch.fwd.astype(np.int64) + ch.bwd
    kept = np.zeros((ch.L, ch.K), dtype=bool)
    for s in range(ch.L):
        for o in range(ch.K):
            kept[s, o] = not any(kept[s, q] and c1[s, q] <= c1[s, o] and xb[s, q] <= xb[s, o]
                                 and need[s, q] <= need[s, o] for q in range(o))
    return kept


def chains():
    return [make_grid_chain(3, 10, 6, 6, M=150), make_grid_chain(4, 7, 5, 4, types=3, M=90),
            make_config_chain(2), make_random_chain(11, 9, 6, allow_zero=True, xmax=2, amax=3, tmax=2)]


def test_kept_set_matches_the_rule():
    for ch in chains():
        h = _handle(ch)
        try:
            kept, k_run = rk.rk_chain_options(h, ch.L, ch.K)
            ref = reference_kept(ch)
            assert np.array_equal(kept, ref), ch.name
            assert k_run == ref.sum(axis=1).max()
            rk.rk_set_option_pruning(h, False)
            kept, k_run = rk.rk_chain_options(h, ch.L, ch.K)
            assert kept.all() and k_run == ch.K
        finally:
            rk.rk_chain_destroy(h)


def test_grid_search_repeats_options():
    """A 20 x 20 budget grid gives fewer than 30 distinct options per block (the paper's
    observation for GPT2); the kept set is exactly the distinct ones here."""
    ch = make_grid_chain(1, 8)
    assert ch.K == 400
    kept = reference_kept(ch)
    for s in range(ch.L):
        distinct = {tuple(v) for v in zip(ch.fwd[s], ch.bwd[s], ch.mem[s], ch.tmp_fwd[s], ch.tmp_bwd[s])}
        assert len(distinct) < 30
        assert kept[s].sum() <= len(distinct)


def test_pruned_chain_keeps_every_value_and_choice():
    """Rebuild each chain from its kept options only (each block's kept options in order,
    padded with copies of its first kept option, which never win) and solve both in the
    oracle: Opt tables equal, and choices equal after mapping option slots back."""
    for ch in chains():
        kept = reference_kept(ch)
        kr = kept.sum(axis=1).max()
        slots = np.array([np.concatenate([np.flatnonzero(r), np.full(kr - r.sum(), np.flatnonzero(r)[0])])
                          for r in kept])
        pick = lambda a: np.ascontiguousarray(np.take_along_axis(a, slots, axis=1)).astype(np.int32)
        small = Chain(L=ch.L, K=int(kr), x=ch.x, fn_time=ch.fn_time, fn_tmp=ch.fn_tmp, fwd=pick(ch.fwd),
                      bwd=pick(ch.bwd), mem=pick(ch.mem), tmp_fwd=pick(ch.tmp_fwd),
                      tmp_bwd=pick(ch.tmp_bwd), M=ch.M, name=ch.name + "-kept")
        full, red = oracle.solve(ch), oracle.solve(small)
        assert np.array_equal(full.opt, red.opt), ch.name
        L = ch.L
        cells = oracle.cell_index(L)
        arg = red.arg.astype(np.int64).copy()
        for s in range(L):
            for t in range(s, L):
                col = arg[:, cells[s, t]]
                opt = col >= L
                col[opt] = L + slots[s][col[opt] - L]
        assert np.array_equal(arg, full.arg.astype(np.int64)), ch.name
