"""rk_solve_noalloc (the fill in the library's static device array, for callers that
cannot allocate) against rk_solve on the same chains: identical answers, Opt and choice
tables and schedules, over two calls in a row, the second with a smaller input."""
import numpy as np
import pytest

import oracle
from paper_2307_01236_amd import rk
from paper_2307_01236_amd.chaingen import make_config_chain, make_random_chain

pytestmark = pytest.mark.gpu


def reference(ch, M):
    s = rk.Solver(ch)
    try:
        ans = s.solve(M)
        opt, arg = s.rows()
        sched = s.schedule() if ans != rk.RK_INF else None
    finally:
        s.close()
    return ans, opt, arg, sched


def noalloc_result(s, M, stream_ptr=None):
    rk.rk_solve_noalloc(s.h, M, stream_ptr)
    s.M = M
    ans = s.result()
    opt, arg = s.rows()
    sched = s.schedule() if ans != rk.RK_INF else None
    return ans, opt, arg, sched


def same(a, b):
    assert a[0] == b[0]
    assert np.array_equal(a[1], b[1]) and np.array_equal(a[2], b[2])
    if a[3] is None:
        assert b[3] is None
    else:
        assert np.array_equal(a[3][0], b[3][0]) and a[3][1] == b[3][1]


def test_noalloc_matches_solve_twice_second_smaller():
    import torch
    ch = make_config_chain(1)  # L=64, K=5, M=1000
    small = make_random_chain(4242, 20, 3)
    s = rk.Solver(ch)
    t = rk.Solver(small)
    try:
        with pytest.raises(rk.RKError) as e:  # not set up on the device yet
            rk.rk_solve_noalloc(s.h, 100)
        assert e.value.code == rk.RK_E_INVAL
        s.solve(10)
        t.solve(5)
        assert rk.rk_workspace_bytes(s.h, 1000) <= rk.RK_NOALLOC_MAX_BYTES
        with pytest.raises(rk.RKError) as e:  # tables larger than the static array
            rk.rk_solve_noalloc(s.h, 20000)
        assert e.value.code == rk.RK_E_NOMEM
        got1 = noalloc_result(s, 1000)
        same(got1, reference(ch, 1000))
        assert got1[0] == oracle.solve(ch, 1000).answer
        got2 = noalloc_result(s, 400)  # a smaller input: fewer budgets
        same(got2, reference(ch, 400))
        st = torch.cuda.Stream()
        got3 = noalloc_result(t, small.M, st.cuda_stream)  # a smaller chain, on a torch stream
        same(got3, reference(small, small.M))
        got4 = noalloc_result(s, 1000)  # back to the first, after another chain used the array
        same(got4, got1)
    finally:
        s.close()
        t.close()
