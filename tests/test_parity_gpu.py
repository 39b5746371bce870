"""Parity of the HIP path with the CPU oracle (MI355X).

Every value compared here comes from the C ABI (librkrotor through its thin
binding) on one side and from the oracle on the other; both get the same
seeded chains.  Opt tables, recorded choices and schedules must match exactly:
all costs are integers.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2307_01236_amd import rk
from paper_2307_01236_amd.chaingen import (CONFIGS, make_config_chain, make_grid_chain,
                                            make_random_chain, relaxations, store_all_bound)

pytestmark = pytest.mark.gpu
INF = rk.RK_INF


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def full_parity(ch, M=None, check_schedule=True, prune=True):
    """Whole Opt and choice tables, the answer and the schedule."""
    M = ch.M if M is None else M
    say(f"  full parity {ch.name} L={ch.L} K={ch.K} M={M} pruning={prune}")
    sol = oracle.solve(ch, M)
    s = rk.Solver(ch)
    try:
        s.set_option_pruning(prune)
        ans = s.solve(M)
        assert ans == sol.answer, (ans, sol.answer)
        g_opt, g_arg = s.rows()
        o_opt, o_arg = sol.rows()
        bad = np.argwhere(g_opt != o_opt)
        assert bad.size == 0, f"Opt differs at {len(bad)} cells, first {bad[:3].tolist()}"
        bad = np.argwhere(g_arg != o_arg)
        assert bad.size == 0, f"choice differs at {len(bad)} cells, first {bad[:3].tolist()}"
        if check_schedule:
            check_same_schedule(s, sol, ch, M)
    finally:
        s.close()
    return sol


def check_same_schedule(s, sol, ch, M):
    exp = oracle.schedule(sol, M)
    if exp is None:
        with pytest.raises(rk.RKError) as e:
            s.schedule()
        assert e.value.code == rk.RK_E_INFEASIBLE
        return
    ops, nfwd = s.schedule()
    assert np.array_equal(ops, exp[0]) and nfwd == exp[1]
    ok, tm, pk, _ = oracle.simulate(ch, ops)
    assert ok and tm == sol.answer and pk <= M


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_configs_full_tables(cfg):
    for rep in range(2 if cfg < 2 else 1):
        full_parity(make_config_chain(cfg, rep))


def test_config0_all_seeds():
    for rep in range(2, 5):
        full_parity(make_config_chain(0, rep))


def fuzz_chains():
    out = []
    rng = np.random.default_rng(12345)
    for seed in range(24):
        L = int(rng.integers(1, 41))
        K = int(rng.integers(1, 17))
        uniform = seed % 4 == 3
        ch = make_random_chain(5000 + seed, L, K, allow_zero=seed % 3 == 0, uniform=uniform,
                               small_times=seed % 2 == 0, xmax=int(rng.integers(1, 12)),
                               amax=int(rng.integers(0, 20)), tmax=int(rng.integers(0, 8)), tmin=0)
        hi = store_all_bound(ch)
        # budgets from nothing to beyond keeping everything, with ragged widths
        M = int(rng.choice([0, 1, hi // 3, hi // 2, hi, 2 * hi + 37, 255, 256, 257]))
        out.append((ch, M))
    return out


@pytest.mark.parametrize("idx", range(24))
def test_fuzz_full_tables(idx):
    ch, M = fuzz_chains()[idx]
    full_parity(ch, M)


@pytest.mark.parametrize("idx", range(4))
def test_longer_random_chains_full_tables(idx):
    """Random (not uniform) chains long enough for band products at spans 32, 64 and 96 and
    for both mid-product levels, including the folds into stored partials (lo > 0)."""
    rng = np.random.default_rng(777 + idx)
    L = int(rng.integers(65, 101))
    K = int(rng.integers(1, 17))
    ch = make_random_chain(9000 + idx, L, K, xmax=int(rng.integers(1, 40)), amax=int(rng.integers(1, 60)),
                           tmax=int(rng.integers(0, 20)), tmin=0, small_times=idx % 2 == 1)
    M = int(rng.integers(store_all_bound(ch) // 4, store_all_bound(ch) + 1))
    full_parity(ch, min(M, 700))


def test_single_block_and_tiny_budgets():
    ch = make_random_chain(77, 1, 4)
    for M in (0, 1, 5, 63, 64, 65, 200):
        full_parity(ch, M)


def test_budget_below_x0_is_infeasible():
    ch = make_config_chain(0)
    s = rk.Solver(ch)
    try:
        assert s.solve(int(ch.x[0]) - 1) == INF
        with pytest.raises(rk.RKError) as e:
            s.schedule()
        assert e.value.code == rk.RK_E_INFEASIBLE
    finally:
        s.close()


def test_resolve_same_chain_different_budgets():
    ch = make_config_chain(1)
    s = rk.Solver(ch)
    try:
        for M in (1000, 400, 1500, 120, 1000):
            sol = oracle.solve(ch, M)
            assert s.solve(M) == sol.answer
            opt, arg = s.rows()
            o_opt, o_arg = sol.rows()
            assert np.array_equal(opt, o_opt) and np.array_equal(arg, o_arg)
    finally:
        s.close()


def test_async_in_torch_workspace_on_torch_stream():
    import torch
    ch = make_config_chain(1)
    sol = oracle.solve(ch)
    s = rk.Solver(ch)
    try:
        nbytes = s.workspace_bytes(ch.M)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
        st = torch.cuda.Stream()
        s.solve_async(ch.M, ws.data_ptr(), nbytes, st.cuda_stream)
        assert s.result() == sol.answer
        opt, arg = s.rows()
        o_opt, o_arg = sol.rows()
        assert np.array_equal(opt, o_opt) and np.array_equal(arg, o_arg)
        check_same_schedule(s, sol, ch, ch.M)
        with pytest.raises(rk.RKError) as e:
            s.solve_async(ch.M, ws.data_ptr(), nbytes - 1, st.cuda_stream)
        assert e.value.code == rk.RK_E_NOMEM
    finally:
        s.close()


def sub_rows_parity(s, ch, s0, n):
    """Rows (s0+a, s0+b) of the full GPU table against the oracle on blocks s0..s0+n-1:
    a span only involves its own blocks, so its row equals the sub-chain's."""
    sub = ch.sub(s0, s0 + n - 1)
    say(f"  sub-chain parity {ch.name} blocks {s0}..{s0 + n - 1}")
    sol = oracle.solve(sub, s.M)
    for a in range(n):
        for b in range(a, n):
            g_opt, g_arg = s.row(s0 + a, s0 + b)
            o_opt, o_arg = sol.opt_row(a, b), sol.arg_row(a, b).astype(np.int32)
            assert np.array_equal(g_opt, o_opt), (s0 + a, s0 + b)
            exp = np.where(o_arg < 0, -1, np.where(o_arg >= n, o_arg - n + ch.L, o_arg + s0))
            assert np.array_equal(g_arg.astype(np.int32), exp), (s0 + a, s0 + b)


def check_properties(ch, opt, M):
    """Whole-table properties that hold at any size: the infeasibility pattern of the
    budget-free recursion, Opt non-increasing in m, and the store-all lower bound."""
    mf = oracle.min_feasible(ch)
    m = np.arange(M + 1)
    assert np.array_equal(opt != INF, m[None, :] >= mf[:, None])
    assert (opt[:, 1:] <= opt[:, :-1]).all()  # INF is INT32_MAX: the int32 order is the order
    top = opt[oracle.cell_index(ch.L)[0, ch.L - 1]]
    lb = (ch.fwd.astype(np.int64) + ch.bwd).min(axis=1).sum()
    assert (top[top != INF] >= lb).all()


def test_config3_full_table_against_oracle():
    """Configuration 3 (L=256, K=8, M=4000: 1.2e10 candidates) at full size: every Opt and
    choice row, the answer and the schedule against the oracle run in this process."""
    ch = make_config_chain(3)
    say(f"  solving {ch.name} on the GPU")
    s = rk.Solver(ch)
    try:
        ans = s.solve()
        g_opt, g_arg = s.rows()
        ops, nfwd = s.schedule()
    finally:
        s.close()
    say("  oracle ...")
    sol = oracle.solve(ch)
    assert ans == sol.answer, (ans, sol.answer)
    o_opt, o_arg = sol.rows()
    cells = oracle.cell_index(ch.L)
    for name, g, o in (("Opt", g_opt, o_opt), ("choice", g_arg, o_arg)):
        bad = np.argwhere(g != o)
        if bad.size:
            k, m = bad[0]
            s_, t_ = map(int, np.argwhere(cells == k)[0])
            raise AssertionError(f"{name} differs at {len(bad)} entries, first (s,t,m)=({s_},{t_},{m}): "
                                 f"GPU {g[k, m]} oracle {o[k, m]}")
    exp_ops, exp_nfwd = oracle.schedule(sol)
    assert np.array_equal(ops, exp_ops) and nfwd == exp_nfwd
    ok, tm, pk, _ = oracle.simulate(ch, ops)
    assert ok and tm == ans and pk <= ch.M
    check_properties(ch, g_opt, ch.M)


def test_config4_full_table_against_oracle_digests():
    """Configuration 4 (L=384, K=16, M=6000: 4.4e8 cells) at full size, in the launch
    configuration the benchmark times: every Opt and choice row against per-row digests of
    the oracle's tables (tests/golden/config4_*, written by make_config_digests.py from the
    oracle alone), the answer and the schedule against the oracle's.  A differing row is
    recomputed by the oracle on its own blocks, which names the first differing (s, t, m)."""
    import json
    import os
    from rowdigest import arg_digests, opt_digests
    gold = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
    with open(os.path.join(gold, "config4_oracle.json")) as f:
        meta = json.load(f)
    dig = np.load(os.path.join(gold, "config4_row_digests.npz"))
    ch = make_config_chain(4)
    assert ch.sha256() == meta["chain_sha256"], "the generator no longer draws the stored chain"
    say(f"  solving {ch.name} on the GPU")
    s = rk.Solver(ch)
    try:
        ans = s.solve()
        g_opt, g_arg = s.rows()
        ops, nfwd = s.schedule()
    finally:
        s.close()
    assert ans == meta["answer"], (ans, meta["answer"])
    god, gad = opt_digests(g_opt), arg_digests(g_arg)
    bad = np.flatnonzero((god != dig["opt"]) | (gad != dig["arg"]))
    if bad.size:
        cells = oracle.cell_index(ch.L)
        spans = [tuple(map(int, np.argwhere(cells == k)[0])) for k in bad]
        s_, t_ = min(spans, key=lambda st: (st[1] - st[0], st[0]))  # the shortest differing span
        k = int(cells[s_, t_])
        sub = oracle.solve(ch.sub(s_, t_))
        o_opt = sub.opt_row(0, t_ - s_)
        o_arg = sub.arg_row(0, t_ - s_).astype(np.int32)
        n = t_ - s_ + 1
        o_arg = np.where(o_arg < 0, -1, np.where(o_arg >= n, o_arg - n + ch.L, o_arg + s_))
        where = np.flatnonzero((g_opt[k] != o_opt) | (g_arg[k].astype(np.int32) != o_arg))
        m = int(where[0]) if where.size else -1
        raise AssertionError(f"{bad.size} rows differ from the oracle's digests; shortest differing span "
                             f"({s_},{t_}), first differing m={m}: GPU Opt/choice "
                             f"{g_opt[k, m]}/{g_arg[k, m]}, oracle {o_opt[m]}/{o_arg[m]}")
    assert np.array_equal(ops, np.asarray(meta["schedule"], dtype=np.int32)) and nfwd == meta["n_fwd"]
    ok, tm, pk, _ = oracle.simulate(ch, ops)
    assert ok and tm == ans and pk <= ch.M
    check_properties(ch, g_opt, ch.M)


def test_profiling_counts_launches():
    ch = make_config_chain(1)
    s = rk.Solver(ch)
    try:
        s.set_profiling(True)
        s.solve()
        stats = s.kernel_stats()
        total = sum(v[0] for v in stats.values())
        ms, launches = s.fill_ms()
        assert total == launches and launches >= 1
        assert sum(v[1] for v in stats.values()) <= ms * 1.05 + 0.05
        # the kernels' relaxation counts add up to the recurrence's candidate count; the
        # evaluated ones leave out tiles past the store-everything budget msa
        assert sum(v[2] for v in stats.values()) == relaxations(ch.L, ch.K, ch.M)
        assert 0 < sum(v[3] for v in stats.values()) < sum(v[2] for v in stats.values())
        for name, v in stats.items():
            assert v[3] <= v[2], (name, v)
            # every fill kernel that runs moves table rows
            assert v[4] % 4 == 0 and (v[4] > 0) == (v[0] > 0 and name != "k_init_inf_rows"), (name, v)
    finally:
        s.close()


@pytest.mark.parametrize("cfg", [1, 2])
def test_profiling_device_counts(cfg):
    """Mode 2 runs the counting variants of the fill kernels: the same launches, results and
    relaxation counts as mode 1, evaluated counts and table bytes at most mode 1's (the
    lower bound only ever skips), the same product and finalize counts on a second solve
    (the counters restart with every fill), and the answer the oracle's."""
    ch = make_config_chain(cfg)
    s = rk.Solver(ch)
    try:
        s.set_profiling(1)
        a1 = s.solve()
        st1 = s.kernel_stats()
        s.set_profiling(2)
        a2 = s.solve()
        st2 = s.kernel_stats()
        a3 = s.solve()
        st3 = s.kernel_stats()
        s.set_profiling(0)
        assert a1 == a2 == a3 == oracle.solve(ch).answer
        assert st1.keys() == st2.keys()
        for name in st1:
            n1, _, w1, e1, b1 = st1[name]
            n2, _, w2, e2, b2 = st2[name]
            assert (n1, w1) == (n2, w2), name
            assert 0 <= e2 <= e1, (name, e1, e2)
            assert 0 <= b2 <= b1 and b2 % 4 == 0, (name, b1, b2)
            assert (e2 > 0) == (e1 > 0) and (b2 > 0) == (b1 > 0), name
            if name == "k_mid":
                # a mid tile's skip test reads partials that the launch's other tiles may be
                # lowering at that moment: its counts may differ from solve to solve
                assert 0 <= st3[name][3] <= e1 and 0 <= st3[name][4] <= b1, name
            else:
                assert st3[name][3:] == st2[name][3:], name
        # from span 64 on, a band product's split ranges pass its 40-split first pass and
        # get cut: fewer candidates than its tiles cover
        if ch.L > 64:
            assert st2["k_product"][3] < st1["k_product"][3]
            assert st2["k_product"][4] < st1["k_product"][4]
    finally:
        s.close()


def test_graph_replays_match_oracle():
    """Repeated solves at one budget replay the captured launch sequence; each replay, with
    other solves and read-backs in between, must still match the oracle exactly."""
    ch, other = make_config_chain(1), make_config_chain(0)
    sol, osol = oracle.solve(ch), oracle.solve(other)
    o_opt, o_arg = sol.rows()
    exp_ops = oracle.schedule(sol)
    s, t = rk.Solver(ch), rk.Solver(other)
    try:
        for rep in range(4):
            say(f"  replay {rep}")
            assert s.solve() == sol.answer
            opt, arg = s.rows(want_arg=rep == 0)
            assert np.array_equal(opt, o_opt)
            if rep == 0:
                assert np.array_equal(arg, o_arg)
            ops, nfwd = s.schedule()
            assert np.array_equal(ops, exp_ops[0]) and nfwd == exp_ops[1]
            assert t.solve() == osol.answer
            s.set_profiling(rep % 2 == 1)  # switching profiling re-captures the sequence
    finally:
        s.close()
        t.close()


def test_tradeoff_curve_matches_oracle():
    """Sec. 4's overhead-against-memory curve from one fill: every budget's optimum, read from
    the table's top row, equals the oracle's; re-solving at a smaller budget agrees."""
    for ch, M in [(make_config_chain(0), None), (make_config_chain(1), None), (make_config_chain(2), None)] + \
            fuzz_chains()[:6]:
        M = ch.M if M is None else M
        sol = oracle.solve(ch, M)
        s = rk.Solver(ch)
        try:
            s.solve(M)
            curve = s.tradeoff_curve().astype(np.int64)
            assert np.array_equal(curve, oracle.tradeoff_curve(sol)), ch.name
            assert np.array_equal(s.tradeoff_curve(min(5, M + 1)), curve[: min(5, M + 1)])
            b = M // 2
            if b >= 0:
                assert s.solve(b) == curve[b]
        finally:
            s.close()


def test_rotor_against_rk_rotor_curves():
    """Rotor (one saving option per block, keep everything) against rk-Rotor's K options on
    the tie-heavy GPT-like workload: the GPU curves equal the oracle's on sampled budgets and
    rk-Rotor's lies on or below Rotor's everywhere."""
    ch = make_config_chain(1)
    rot_ch = ch.options([0])
    curves = []
    for c in (ch, rot_ch):
        s = rk.Solver(c)
        try:
            s.solve(c.M)
            curves.append(s.tradeoff_curve().astype(np.int64))
        finally:
            s.close()
        sol = oracle.solve(c)
        assert np.array_equal(curves[-1], oracle.tradeoff_curve(sol)), c.name
    rkc, rot = curves
    assert (rot >= rkc).all()
    assert np.argmax(rkc < INF) <= np.argmax(rot < INF)


def test_tradeoff_curve_errors():
    ch = make_config_chain(0)
    s = rk.Solver(ch)
    try:
        with pytest.raises(rk.RKError) as e:
            s.M = ch.M
            s.tradeoff_curve()
        assert e.value.code == rk.RK_E_NOT_SOLVED
        s.solve(ch.M)
        with pytest.raises(rk.RKError) as e:
            s.tradeoff_curve(ch.M + 2)
        assert e.value.code == rk.RK_E_INVAL
        assert s.tradeoff_curve(0).size == 0
    finally:
        s.close()


@pytest.mark.parametrize("prune", [True, False])
def test_grid_options_pruned_and_unpruned(prune):
    """An emulated budget-grid option search (100 options per block, mostly repeats, three
    block types): with pruning the kernels evaluate only the distinct options; tables,
    choices (in the caller's option indices) and the schedule match the oracle exactly
    either way."""
    ch = make_grid_chain(5, 24, 10, 10, types=3)
    full_parity(ch, prune=prune)


def test_pruning_switch_between_solves():
    """Turning pruning off and on between solves of one chain rebuilds the device arrays and
    the captured launch sequence; every solve still matches the oracle."""
    ch = make_grid_chain(6, 20, 8, 8)
    sol = oracle.solve(ch)
    o_opt, o_arg = sol.rows()
    exp = oracle.schedule(sol)
    s = rk.Solver(ch)
    try:
        for prune in (True, False, True):
            s.set_option_pruning(prune)
            assert s.solve() == sol.answer
            opt, arg = s.rows()
            assert np.array_equal(opt, o_opt) and np.array_equal(arg, o_arg), prune
            ops, nfwd = s.schedule()
            assert np.array_equal(ops, exp[0]) and nfwd == exp[1]
            kept, k_run = s.options()
            assert (k_run < ch.K) == prune
    finally:
        s.close()


def test_backtrace_with_option_sizes_in_global_memory():
    """400 options per block on 36 blocks, pruning off: L*K = 14400 option sizes do not fit the
    backtrace's LDS copy, so it reads them from global memory, and a visited cell's options
    take seven rounds of lanes.  Tables and schedule still match the oracle exactly."""
    ch = make_grid_chain(8, 36, 20, 20)
    full_parity(ch, prune=False)


def test_longest_chain():
    """RK_MAX_L = 2000 blocks (1999 finalize launches; a backtrace whose LDS stack of up to
    2L + 8 frames and x copy take 72 KB).  Exact parity on sub-chains at both ends; the
    schedule replays legally in the oracle's simulator at exactly the answer and within the
    budget (the oracle's full table would take minutes; the simulator shares nothing with it)."""
    L = rk.RK_MAX_L
    ch = make_random_chain(2024, L, 2, M=600, xmax=3, amax=4, tmax=2, small_times=True)
    s = rk.Solver(ch)
    try:
        ans = s.solve()
        assert ans != INF
        for s0 in (0, L - 14):
            sub_rows_parity(s, ch, s0, 14)
        ops, nfwd = s.schedule()
        ok, tm, pk, bad = oracle.simulate(ch, ops)
        assert ok, bad
        assert tm == ans and pk <= ch.M
        assert ops[nfwd][0] == rk.RK_BWD
    finally:
        s.close()


def test_fill_inside_a_torch_graph_capture():
    """The caller captures rk_solve_async into its own graph (torch.cuda.graph) after one eager
    solve set the chain up.  Each replay refills the table from scratch: between replays the
    workspace is overwritten with zeros and other eager work runs, and every replay's answer,
    table and schedule must still match the oracle."""
    import torch
    ch = make_config_chain(1)
    sol = oracle.solve(ch)
    o_opt, o_arg = sol.rows()
    exp = oracle.schedule(sol)
    s = rk.Solver(ch)
    try:
        nbytes = s.workspace_bytes(ch.M)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
        st = torch.cuda.Stream()
        s.solve_async(ch.M, ws.data_ptr(), nbytes, st.cuda_stream)  # eager: uploads the chain
        assert s.result() == sol.answer
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=st):
            s.solve_async(ch.M, ws.data_ptr(), nbytes, st.cuda_stream)
        other = torch.randn(1 << 20, device="cuda:0")
        for rep in range(3):
            ws.zero_()
            other.mul_(1.5)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            say(f"  replay {rep}")
            assert s.result() == sol.answer
            opt, arg = s.rows(want_arg=rep == 0)
            assert np.array_equal(opt, o_opt), rep
            if rep == 0:
                assert np.array_equal(arg, o_arg)
            ops, nfwd = s.schedule()
            assert np.array_equal(ops, exp[0]) and nfwd == exp[1]
        # a fill inside the caller's graph has no timing; an eager solve afterwards has
        with pytest.raises(rk.RKError) as e:
            s.fill_ms()
        assert e.value.code == rk.RK_E_INVAL
        s.solve_async(ch.M, ws.data_ptr(), nbytes, st.cuda_stream)
        assert s.result() == sol.answer and s.fill_ms()[0] > 0
    finally:
        s.close()


def test_option_sizes_beyond_the_staged_halo():
    """Options that keep up to 700 slots: case 1's shift exceeds the 256 columns the finalize
    stages in LDS, so it reads the shifted row from global memory.  Full-table parity."""
    ch = make_random_chain(4242, 40, 4, xmax=40, amax=700, tmax=60, tmin=0)
    assert int(ch.mem.max()) + int(ch.x.max()) > 256
    full_parity(ch, 3000)


@pytest.mark.parametrize("idx", range(8))
def test_medium_random_chains_sampled(idx):
    """Random chains of 110-260 blocks (several bands, ragged band and column tails), 1-24
    options, budgets 300-2500: exact parity on three sampled sub-chains, and on the whole
    table the infeasibility pattern, monotonicity in m and a schedule that replays at the
    answer."""
    rng = np.random.default_rng(4100 + idx)
    L = int(rng.integers(110, 261))
    K = int(rng.integers(1, 25))
    ch = make_random_chain(4100 + idx, L, K, xmax=int(rng.integers(1, 30)), amax=int(rng.integers(1, 80)),
                           tmax=int(rng.integers(0, 30)), tmin=0, small_times=idx % 2 == 0,
                           allow_zero=idx % 3 == 0)
    M = int(rng.integers(300, 2501))
    say(f"  medium chain L={L} K={K} M={M}")
    s = rk.Solver(ch)
    try:
        ans = s.solve(M)
        for s0, n in ((0, 16), (int(rng.integers(1, L - 16)), 16), (L - 16, 16)):
            sub_rows_parity(s, ch, s0, n)
        mf = oracle.min_feasible(ch)
        cells = oracle.cell_index(L)
        m = np.arange(M + 1)
        for _ in range(30):
            a = int(rng.integers(0, L))
            b = int(rng.integers(a, L))
            row, _ = s.row(a, b, want_arg=False)
            assert np.array_equal(row != INF, m >= mf[cells[a, b]]), (a, b)
            r64 = row.astype(np.int64)
            assert (r64[1:] <= r64[:-1]).all(), (a, b)
        if ans != INF:
            ops, nfwd = s.schedule()
            ok, tm, pk, bad = oracle.simulate(ch, ops)
            assert ok and tm == ans and pk <= M, (ok, tm, ans, pk, bad)
    finally:
        s.close()


@pytest.mark.parametrize("M", [24998, 25000])
def test_mid_levels_at_large_budgets(M):
    """64 blocks at about 25 000 budget columns (1.6e6 blocks x budget columns) with shifts of
    up to 50 columns: mid products of widths 16 and 8 and a finalize that covers the splits
    whose longer operand spans the last 8 spans.  Full-table parity."""
    ch = make_random_chain(6464, 64, 3, xmax=50, amax=400, tmax=100, tmin=0)
    sol = full_parity(ch, M)
    assert sol.answer != INF
    s = rk.Solver(ch)
    try:
        s.set_profiling(True)
        s.solve(M)
        stats = s.kernel_stats()
        n_mid = stats["k_mid"][0]
        # the kernels' relaxation counts still add up to the recurrence's candidate count
        assert sum(v[2] for v in stats.values()) == relaxations(ch.L, ch.K, M)
    finally:
        s.close()
    # mids of width 16 at d = 16, 48 and of width 8 at d = 8, 24, 40, 56
    assert n_mid == 6, n_mid


@pytest.mark.parametrize("seed", [97003, 97008])
def test_several_bands_at_large_tables(seed):
    """Chains of 64-110 blocks with at least 1.6e6 blocks x budget columns (78 and 105
    blocks, one option): two or three band products, mids of widths 16 and 8, and shifts
    of up to a few hundred columns.  Full-table parity."""
    rng = np.random.default_rng(seed)
    L = int(rng.integers(64, 110))
    K = int(rng.integers(1, 4))
    M = int(rng.integers(1_600_000 // L, 1_600_000 // L + 3000))
    ch = make_random_chain(seed, L, K, M=M, xmax=int(rng.integers(1, 300)), amax=int(rng.integers(1, 1500)),
                           tmax=int(rng.integers(0, 300)), tmin=0, allow_zero=bool(rng.integers(0, 2)),
                           small_times=bool(rng.integers(0, 2)))
    assert ch.L * (M + 1) >= 1_600_000
    full_parity(ch, M)


def test_wide_budget():
    """200 001 budget columns on a short chain with large sizes: a left pad of ~2000 columns,
    1 563 column chunks per cell in the finalize and shifts far beyond its staged halo.
    Full-table parity."""
    ch = make_random_chain(777, 12, 3, xmax=2000, amax=9000, tmax=3000, tmin=0)
    full_parity(ch, 200000)
