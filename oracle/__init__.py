"""CPU oracle of the rk-Rotor dynamic program -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow reference that the HIP path is checked
against.  Only the tests, the package smoke check and the benchmark's CPU
baseline may import it; the solver library never does, and it shares no code
with it.  ``build()`` compiles ``rko.c`` with gcc into ``librko.so`` next to
this file; the wrappers below only marshal arguments.

Tables returned here are in the oracle's own layout: m-major,
``opt[m, cell(s,t)]`` with cells in upper-triangle row-major order.
``rows()`` turns them into an [ncells, M+1] array in that same cell order.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "librko.so")
INF = 2**31 - 1

FWD_NOSAVE, FWD_SAVE, BWD, FREE_X, REFWD = 0, 1, 2, 3, 4
OK, E_INVAL, E_INFEASIBLE, E_BUFSZ, E_REPLAY = 0, -1, -6, -7, -8


def build(force: bool = True) -> str:
    src = os.path.join(HERE, "rko.c")
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(src):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-Werror", "-shared",
                               "-fPIC", src, "-o", tmp])
        os.replace(tmp, LIB)
    return LIB


class _Chain(C.Structure):
    _fields_ = [("L", C.c_int32), ("K", C.c_int32)] + [
        (n, C.POINTER(C.c_int32))
        for n in ("x", "fn_time", "fn_tmp", "fwd", "bwd", "mem", "tmp_fwd", "tmp_bwd", "refwd")]


class _Op(C.Structure):
    _fields_ = [("kind", C.c_int32), ("block", C.c_int32), ("option", C.c_int32)]


class Library:
    """ctypes view of one build of the oracle (the default one, or a test's variant)."""

    def __init__(self, path: str):
        lib = C.CDLL(path)
        P = C.POINTER
        lib.rko_ncells.argtypes = [C.c_int32]
        lib.rko_ncells.restype = C.c_int64
        lib.rko_cell.argtypes = [C.c_int32, C.c_int32, C.c_int32]
        lib.rko_cell.restype = C.c_int64
        lib.rko_solve.argtypes = [P(_Chain), C.c_int32, P(C.c_int32), P(C.c_int16), P(C.c_int32),
                                  P(C.c_int16), P(C.c_int32)]
        lib.rko_schedule.argtypes = [P(_Chain), C.c_int32, P(C.c_int16), P(C.c_int16), P(_Op), C.c_int64,
                                     P(C.c_int64), P(C.c_int64)]
        lib.rko_simulate.argtypes = [P(_Chain), P(_Op), C.c_int64, P(C.c_int64), P(C.c_int64),
                                     P(C.c_int64)]
        lib.rko_min_feasible.argtypes = [P(_Chain), P(C.c_int64)]
        for f in (lib.rko_solve, lib.rko_schedule, lib.rko_simulate, lib.rko_min_feasible):
            f.restype = C.c_int
        self.lib = lib
        self.path = path


_default = None


def _load(lib: "Library | None" = None):
    global _default
    if lib is not None:
        return lib.lib
    if _default is None:
        if not os.path.exists(LIB):
            build(force=False)
        _default = Library(LIB)
    return _default.lib


def build_variant(src: str, out: str) -> "Library":
    """Compile another copy of the oracle source (used by the mutation tests)."""
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-w", "-shared", "-fPIC", "-I", HERE, src,
                           "-o", out])
    return Library(out)


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


class _Bound:
    """Keeps the int32 copies alive while the C struct points at them.  A chain with a
    `refwd` array (not None) switches on the saving sweep (rko.h)."""

    def __init__(self, ch):
        self.arrs = [np.ascontiguousarray(a, dtype=np.int32).ravel() for a in ch.arrays()]
        rf = getattr(ch, "refwd", None)
        self.refwd = None if rf is None else np.ascontiguousarray(rf, dtype=np.int32).ravel()
        self.s = _Chain(ch.L, ch.K, *[_i32p(a) for a in self.arrs],
                        _i32p(self.refwd) if self.refwd is not None else None)


def ncells(L: int) -> int:
    return L * (L + 1) // 2


def cell(L: int, s: int, t: int) -> int:
    return int(_load().rko_cell(L, s, t))


def cell_index(L: int) -> np.ndarray:
    """[L, L] array: cell(s,t) for t >= s, -1 elsewhere."""
    idx = -np.ones((L, L), dtype=np.int64)
    k = 0
    for s in range(L):
        for t in range(s, L):
            idx[s, t] = k
            k += 1
    return idx


class Solution:
    def __init__(self, ch, M, opt, arg, answer, hval=None, harg=None):
        self.chain, self.M, self.opt, self.arg, self.answer = ch, M, opt, arg, answer
        self.hval, self.harg = hval, harg  # the saving sweep's H table and choices, or None
        self.cells = cell_index(ch.L)

    def opt_row(self, s: int, t: int) -> np.ndarray:
        return self.opt[:, self.cells[s, t]]

    def arg_row(self, s: int, t: int) -> np.ndarray:
        return self.arg[:, self.cells[s, t]]

    def rows(self):
        """(opt, arg) as [ncells, M+1] arrays, cells in upper-triangle row-major order."""
        return np.ascontiguousarray(self.opt.T), np.ascontiguousarray(self.arg.T)

    def h_rows(self):
        """(hval, harg) of the saving sweep as [ncells, M+1] arrays (same order)."""
        return np.ascontiguousarray(self.hval.T), np.ascontiguousarray(self.harg.T)


def solve(ch, M: int | None = None, lib: Library | None = None) -> Solution:
    lib = _load(lib)
    M = ch.M if M is None else int(M)
    n = ncells(ch.L)
    opt = np.empty((M + 1, n), dtype=np.int32)
    arg = np.empty((M + 1, n), dtype=np.int16)
    ans = C.c_int32(0)
    b = _Bound(ch)
    hval = harg = None
    if b.refwd is not None:
        hval = np.empty((M + 1, n), dtype=np.int32)
        harg = np.empty((M + 1, n), dtype=np.int16)
    i16 = C.POINTER(C.c_int16)
    rc = lib.rko_solve(C.byref(b.s), M, _i32p(opt), arg.ctypes.data_as(i16),
                       None if hval is None else _i32p(hval),
                       None if harg is None else harg.ctypes.data_as(i16), C.byref(ans))
    if rc != OK:
        raise ValueError(f"rko_solve failed: {rc}")
    return Solution(ch, M, opt, arg, int(ans.value), hval, harg)


def tradeoff_curve(sol: Solution, n: int | None = None) -> np.ndarray:
    """Best schedule time at each total budget b = 0..n-1 (default n = M+1): the answer of
    the solve at budget b, Opt(0, L-1, b - x_0), INF below x_0 (Sec. 4's overhead-against-
    memory comparison reads this curve).  A fill at M holds every smaller budget's answer,
    because Opt(s, t, m) does not depend on the largest budget filled."""
    ch = sol.chain
    n = sol.M + 1 if n is None else int(n)
    assert 0 <= n <= sol.M + 1
    x0 = int(ch.x[0])
    out = np.full(n, INF, dtype=np.int64)
    if n > x0:
        out[x0:] = sol.opt_row(0, ch.L - 1)[: n - x0]
    return out


def schedule(sol: Solution, M: int | None = None, lib: Library | None = None):
    """Alg. 3 for budget M (default: the solve's M).  Returns (ops[n,3], n_fwd) or None."""
    lib = _load(lib)
    ch = sol.chain
    M = sol.M if M is None else int(M)
    assert M <= sol.M
    b = _Bound(ch)
    # the choice table is laid out for the solve's width; it holds all m <= sol.M
    argp = sol.arg.ctypes.data_as(C.POINTER(C.c_int16))
    hargp = None if sol.harg is None else sol.harg.ctypes.data_as(C.POINTER(C.c_int16))
    nops, nfwd = C.c_int64(0), C.c_int64(0)
    rc = lib.rko_schedule(C.byref(b.s), M, argp, hargp, None, 0, C.byref(nops), C.byref(nfwd))
    if rc == E_INFEASIBLE:
        return None
    if rc != E_BUFSZ:
        raise ValueError(f"rko_schedule sizing failed: {rc}")
    ops = (_Op * max(1, nops.value))()
    rc = lib.rko_schedule(C.byref(b.s), M, argp, hargp, ops, nops.value, C.byref(nops), C.byref(nfwd))
    if rc != OK:
        raise ValueError(f"rko_schedule failed: {rc}")
    out = np.array([(o.kind, o.block, o.option) for o in ops[:nops.value]], dtype=np.int32)
    return out.reshape(-1, 3), int(nfwd.value)


def simulate(ch, ops, lib: Library | None = None) -> tuple[bool, int, int, int]:
    """Replay ops ([n,3] int array).  Returns (ok, time, peak, bad_index)."""
    lib = _load(lib)
    ops = np.ascontiguousarray(np.asarray(ops, dtype=np.int32).reshape(-1, 3))
    b = _Bound(ch)
    tm, pk, bad = C.c_int64(0), C.c_int64(0), C.c_int64(0)
    rc = lib.rko_simulate(C.byref(b.s), ops.ctypes.data_as(C.POINTER(_Op)), len(ops), C.byref(tm),
                          C.byref(pk), C.byref(bad))
    if rc not in (OK, E_REPLAY):
        raise ValueError(f"rko_simulate failed: {rc}")
    return rc == OK, int(tm.value), int(pk.value), int(bad.value)


def min_feasible(ch, lib: Library | None = None) -> np.ndarray:
    """[ncells] smallest budget beyond x_s at which each span is feasible."""
    lib = _load(lib)
    out = np.empty(ncells(ch.L), dtype=np.int64)
    b = _Bound(ch)
    rc = lib.rko_min_feasible(C.byref(b.s), out.ctypes.data_as(C.POINTER(C.c_int64)))
    if rc != OK:
        raise ValueError(f"rko_min_feasible failed: {rc}")
    return out
