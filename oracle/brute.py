"""Exhaustive checks of the rk-Rotor oracle on tiny chains -- TEST INFRASTRUCTURE ONLY.

Two searches that do not use the dynamic program at all:

* ``decision_trees`` enumerates every schedule of the shape rk-Rotor can
  produce (App. C: at each span either case 1 with some option o, or case 2
  with some split i, recursively; with a chain's ``refwd`` also the saving
  sweep with option o and split i, see rko.h), turns each into its operation
  list the way Alg. 3 lays it out, and replays it in the oracle's simulator.  The cheapest
  replay whose peak fits a budget must equal the dynamic program's value at
  that budget, for every budget: this pins the recurrence, its validity
  conditions and its memory accounting at once.

* ``dijkstra_lower_bound`` searches all legal operation orders (any forward,
  backward or forget the simulator accepts, not only rk-Rotor's shapes).  Its
  optimum can only be at most the dynamic program's: the paper notes that
  rk-Rotor does not explore every schedule (Sec. 3.4, sub-optimality).
"""
from __future__ import annotations

import heapq
import itertools

import numpy as np

from . import BWD, FREE_X, FWD_NOSAVE, FWD_SAVE, INF, REFWD, simulate


def _trees(L, K, s, t, memo, sweep=False):
    key = (s, t)
    if key in memo:
        return memo[key]
    out = []
    for o in range(K):
        if s == t:
            out.append(("o", s, o, None))
        else:
            for sub in _trees(L, K, s + 1, t, memo, sweep):
                out.append(("o", s, o, sub))
    for i in range(s + 1, t + 1):
        for right, left in itertools.product(_trees(L, K, i, t, memo, sweep),
                                             _trees(L, K, s, i - 1, memo, sweep)):
            out.append(("i", s, i, (right, left)))
    if sweep:  # F_s^o, sweep s+1..i-1 to x_i, i..t, x_{s+1} again from F_s^o's data, s+1..i-1, B_s^o
        for o in range(K):
            for i in range(s + 2, t + 1):
                for right, left in itertools.product(_trees(L, K, i, t, memo, sweep),
                                                     _trees(L, K, s + 1, i - 1, memo, sweep)):
                    out.append(("h", s, (o, i), (right, left)))
    memo[key] = out
    return out


def _ops(tree, acc):
    kind, s, v, sub = tree
    if kind == "o":
        acc.append((FWD_SAVE, s, v))
        if sub is not None:
            _ops(sub, acc)
        acc.append((BWD, s, v))
    elif kind == "h":
        o, i = v
        right, left = sub
        acc.append((FWD_SAVE, s, o))
        for k in range(s + 1, i):
            acc.append((FWD_NOSAVE, k, -1))
            acc.append((FREE_X, k, -1))
        _ops(right, acc)
        acc.append((FREE_X, i, -1))
        acc.append((REFWD, s, o))
        _ops(left, acc)
        acc.append((BWD, s, o))
    else:
        i = v
        right, left = sub
        acc.append((FWD_NOSAVE, s, -1))
        for k in range(s + 1, i):
            acc.append((FWD_NOSAVE, k, -1))
            acc.append((FREE_X, k, -1))
        _ops(right, acc)
        acc.append((FREE_X, i, -1))
        _ops(left, acc)
    return acc


def count_trees(L: int, K: int, sweep: bool = False) -> int:
    return len(_trees(L, K, 0, L - 1, {}, sweep))


def decision_trees(ch, Mmax: int, lib=None) -> np.ndarray:
    """best[M] for M = 0..Mmax: cheapest rk-Rotor-shaped schedule with peak <= M (INF if none).
    A chain with a ``refwd`` array also gets the saving sweep's trees."""
    best = np.full(Mmax + 1, INF, dtype=np.int64)
    sweep = getattr(ch, "refwd", None) is not None
    for tree in _trees(ch.L, ch.K, 0, ch.L - 1, {}, sweep):
        ops = _ops(tree, [])
        ok, tm, pk, _ = simulate(ch, ops, lib=lib)
        assert ok, "an rk-Rotor-shaped schedule must always replay legally"
        if pk <= Mmax:
            best[pk:] = np.minimum(best[pk:], tm)
    return best


def dijkstra_lower_bound(ch, M: int) -> int:
    """Cheapest legal operation order with every operation's peak <= M (INF if none).  With
    a chain's ``refwd``, making x_{k+1} again from F_k^o's kept data is one more move."""
    L, K = ch.L, ch.K
    refwd = getattr(ch, "refwd", None)
    x = [int(v) for v in ch.x]
    mem = ch.mem.astype(np.int64)
    if x[0] > M:
        return INF
    # state: (bitmask of live x_1..x_L, tuple of kept option per block (-1 none), g)
    # where g is the smallest block index whose output gradient is known (grad_g ready).
    start = (0, tuple([-1] * L), L)

    def used(state):
        xm, h, _ = state
        u = x[0]
        for k in range(1, L + 1):
            if xm >> k & 1:
                u += x[k]
        for k in range(L):
            if h[k] >= 0:
                u += int(mem[k, h[k]])
        return u

    def live(xm, k):
        return k == 0 or (xm >> k & 1)

    dist = {start: 0}
    pq = [(0, start)]
    while pq:
        dcur, st = heapq.heappop(pq)
        if dist.get(st, None) != dcur:
            continue
        xm, h, g = st
        if g == 0 and xm == 0 and all(v < 0 for v in h):
            return dcur
        u = used(st)
        nxt = []
        for k in range(L):
            if live(xm, k) and not live(xm, k + 1):
                if u + x[k + 1] + int(ch.fn_tmp[k]) <= M:
                    nxt.append((int(ch.fn_time[k]), (xm | 1 << (k + 1), h, g)))
                if refwd is not None and h[k] >= 0:
                    o = h[k]
                    if u + x[k + 1] + int(ch.tmp_fwd[k, o]) <= M:
                        nxt.append((int(refwd[k, o]), (xm | 1 << (k + 1), h, g)))
                if h[k] < 0:
                    for o in range(K):
                        if u + x[k + 1] + int(mem[k, o]) + int(ch.tmp_fwd[k, o]) <= M:
                            h2 = list(h)
                            h2[k] = o
                            nxt.append((int(ch.fwd[k, o]), (xm | 1 << (k + 1), tuple(h2), g)))
        if g > 0:
            k = g - 1
            o = h[k]
            if o >= 0 and live(xm, k) and live(xm, k + 1) and u + int(ch.tmp_bwd[k, o]) <= M:
                h2 = list(h)
                h2[k] = -1
                nxt.append((int(ch.bwd[k, o]), (xm & ~(1 << (k + 1)), tuple(h2), k)))
        for k in range(1, L + 1):
            if xm >> k & 1:
                nxt.append((0, (xm & ~(1 << k), h, g)))
        for w, s2 in nxt:
            nd = dcur + w
            if nd < dist.get(s2, INF + 1):
                dist[s2] = nd
                heapq.heappush(pq, (nd, s2))
    return INF
