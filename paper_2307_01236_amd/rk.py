"""Python binding of librkrotor (include/rk.h): argument marshalling only.

Every step of the solve runs in the HIP library.  The functions keep the C
names; non-OK return codes raise ``RKError``.  If ``librkrotor.so`` has not
been built, loading raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librkrotor.so")

RK_INF = 2**31 - 1
RK_TIME_LIMIT = (1 << 30) - 2
RK_MAX_L = 2000
RK_MAX_M = (1 << 26) - 2
RK_FWD_NOSAVE, RK_FWD_SAVE, RK_BWD, RK_FREE_X, RK_REFWD = 0, 1, 2, 3, 4
(RK_OK, RK_E_INVAL, RK_E_OVERFLOW, RK_E_NOMEM, RK_E_DEVICE, RK_E_NOT_SOLVED, RK_E_INFEASIBLE,
 RK_E_BUFSZ, RK_E_INTERNAL) = 0, -1, -2, -3, -4, -5, -6, -7, -8

EXPORTS = ("rk_chain_create", "rk_chain_destroy", "rk_workspace_bytes", "rk_solve", "rk_solve_async",
           "rk_result", "rk_extract_schedule", "rk_read_row", "rk_tradeoff_curve", "rk_last_fill_ms",
           "rk_set_profiling", "rk_set_option_pruning", "rk_chain_options",
           "rk_fill_kernel_stats", "rk_strerror", "rk_solve_noalloc", "rk_chain_set_saving_sweep")
RK_NOALLOC_MAX_BYTES = 64 << 20


class RKError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {rk_strerror(code)} ({code})")


class rk_op(C.Structure):
    _fields_ = [("kind", C.c_int32), ("block", C.c_int32), ("option", C.c_int32)]


_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2307_01236_amd.build.build()")
        # torch ships its own HIP runtime (same soname as the system one).  Loading it first
        # makes the library bind to that copy, so torch's memory and streams and the
        # library's kernels live in one runtime; two runtimes in one process cannot share
        # the GPU.
        import torch  # noqa: F401
        lib = C.CDLL(LIB_PATH)
        P, i32, i64 = C.POINTER, C.c_int32, C.c_int64
        i32p = P(C.c_int32)
        lib.rk_chain_create.argtypes = [i32, i32] + [i32p] * 8 + [P(C.c_void_p)]
        lib.rk_chain_destroy.argtypes = [C.c_void_p]
        lib.rk_chain_destroy.restype = None
        lib.rk_workspace_bytes.argtypes = [C.c_void_p, i32, P(C.c_size_t)]
        lib.rk_solve.argtypes = [C.c_void_p, i32, i32p]
        lib.rk_solve_async.argtypes = [C.c_void_p, i32, C.c_void_p, C.c_size_t, C.c_void_p]
        lib.rk_solve_noalloc.argtypes = [C.c_void_p, i32, C.c_void_p]
        lib.rk_chain_set_saving_sweep.argtypes = [C.c_void_p, i32p]
        lib.rk_result.argtypes = [C.c_void_p, i32p]
        lib.rk_extract_schedule.argtypes = [C.c_void_p, P(rk_op), i64, P(i64), P(i64)]
        lib.rk_read_row.argtypes = [C.c_void_p, i32, i32, i32p, P(C.c_int16)]
        lib.rk_tradeoff_curve.argtypes = [C.c_void_p, i32p, i64]
        lib.rk_last_fill_ms.argtypes = [C.c_void_p, P(C.c_float), i32p]
        lib.rk_set_profiling.argtypes = [C.c_void_p, i32]
        lib.rk_set_option_pruning.argtypes = [C.c_void_p, i32]
        lib.rk_chain_options.argtypes = [C.c_void_p, i32p, i32p]
        lib.rk_fill_kernel_stats.argtypes = [C.c_void_p, i32, i32p, P(C.c_char_p), i32p,
                                             P(C.c_float), P(i64), P(i64), P(i64)]
        lib.rk_strerror.argtypes = [C.c_int]
        lib.rk_strerror.restype = C.c_char_p
        for n in EXPORTS:
            if n not in ("rk_chain_destroy", "rk_strerror"):
                getattr(lib, n).restype = C.c_int
        _lib = lib
    return _lib


def rk_strerror(code: int) -> str:
    return load().rk_strerror(int(code)).decode()


def _check(rc: int, where: str) -> None:
    if rc != RK_OK:
        raise RKError(rc, where)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.int32).ravel()


def rk_chain_create(L, K, x, fn_time, fn_tmp, fwd, bwd, mem, tmp_fwd, tmp_bwd) -> C.c_void_p:
    arrs = [_i32(a) for a in (x, fn_time, fn_tmp, fwd, bwd, mem, tmp_fwd, tmp_bwd)]
    sizes = [L + 1, L, L] + [L * K] * 5
    for a, n in zip(arrs, sizes):
        if a.size != n:
            raise RKError(RK_E_INVAL, "rk_chain_create (array size)")
    h = C.c_void_p()
    ptrs = [a.ctypes.data_as(C.POINTER(C.c_int32)) for a in arrs]
    _check(load().rk_chain_create(int(L), int(K), *ptrs, C.byref(h)), "rk_chain_create")
    return h


def rk_chain_destroy(h) -> None:
    load().rk_chain_destroy(h)


def rk_workspace_bytes(h, M: int) -> int:
    out = C.c_size_t(0)
    _check(load().rk_workspace_bytes(h, int(M), C.byref(out)), "rk_workspace_bytes")
    return int(out.value)


def rk_solve(h, M: int) -> int:
    out = C.c_int32(0)
    _check(load().rk_solve(h, int(M), C.byref(out)), "rk_solve")
    return int(out.value)


def rk_solve_async(h, M: int, workspace_ptr: int, ws_bytes: int, stream_ptr: int | None) -> None:
    _check(load().rk_solve_async(h, int(M), C.c_void_p(workspace_ptr), C.c_size_t(ws_bytes),
                                 C.c_void_p(stream_ptr or 0)), "rk_solve_async")


def rk_chain_set_saving_sweep(h, refwd) -> None:
    """refwd: [L, K] re-forward times (the saving sweep on) or None (off)."""
    if refwd is None:
        _check(load().rk_chain_set_saving_sweep(h, None), "rk_chain_set_saving_sweep")
    else:
        a = _i32(refwd)
        _check(load().rk_chain_set_saving_sweep(h, a.ctypes.data_as(C.POINTER(C.c_int32))),
               "rk_chain_set_saving_sweep")


def rk_solve_noalloc(h, M: int, stream_ptr: int | None = None) -> None:
    _check(load().rk_solve_noalloc(h, int(M), C.c_void_p(stream_ptr or 0)), "rk_solve_noalloc")


def rk_result(h) -> int:
    out = C.c_int32(0)
    _check(load().rk_result(h, C.byref(out)), "rk_result")
    return int(out.value)


def rk_extract_schedule(h):
    """(ops as an [n, 3] int32 array of (kind, block, option), n_fwd)."""
    lib = load()
    n, nf = C.c_int64(0), C.c_int64(0)
    rc = lib.rk_extract_schedule(h, None, 0, C.byref(n), C.byref(nf))
    if rc != RK_E_BUFSZ:
        _check(rc, "rk_extract_schedule")
    buf = (rk_op * max(1, n.value))()
    _check(lib.rk_extract_schedule(h, buf, n.value, C.byref(n), C.byref(nf)), "rk_extract_schedule")
    out = np.frombuffer(buf, dtype=np.int32, count=3 * n.value).reshape(-1, 3).copy()
    return out, int(nf.value)


def rk_read_row(h, s: int, t: int, W: int, want_arg: bool = True):
    opt = np.empty(W, dtype=np.int32)
    arg = np.empty(W, dtype=np.int16) if want_arg else None
    _check(load().rk_read_row(h, int(s), int(t), opt.ctypes.data_as(C.POINTER(C.c_int32)),
                              arg.ctypes.data_as(C.POINTER(C.c_int16)) if want_arg else None),
           "rk_read_row")
    return opt, arg


def rk_tradeoff_curve(h, n: int) -> np.ndarray:
    times = np.empty(max(int(n), 0), dtype=np.int32)
    _check(load().rk_tradeoff_curve(h, times.ctypes.data_as(C.POINTER(C.c_int32)), int(n)),
           "rk_tradeoff_curve")
    return times


def rk_last_fill_ms(h):
    ms, n = C.c_float(0), C.c_int32(0)
    _check(load().rk_last_fill_ms(h, C.byref(ms), C.byref(n)), "rk_last_fill_ms")
    return float(ms.value), int(n.value)


def rk_set_option_pruning(h, enable: bool) -> None:
    _check(load().rk_set_option_pruning(h, 1 if enable else 0), "rk_set_option_pruning")


def rk_chain_options(h, L: int, K: int):
    """(kept [L, K] bool, k_run): which options the solver evaluates, and slots per block."""
    kept = np.empty(L * K, dtype=np.int32)
    kr = C.c_int32(0)
    _check(load().rk_chain_options(h, kept.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(kr)),
           "rk_chain_options")
    return kept.reshape(L, K).astype(bool), int(kr.value)


def rk_set_profiling(h, mode) -> None:
    """mode: False/0 off, True/1 per-launch timing, 2 timing and the device candidate counts."""
    _check(load().rk_set_profiling(h, int(mode)), "rk_set_profiling")


def rk_fill_kernel_stats(h):
    """{kernel name: (launches, summed device ms, relaxations of the recurrence, relaxations
    evaluated, compulsory bytes)} for the last solve."""
    lib = load()
    nk = C.c_int32(0)
    lib.rk_fill_kernel_stats(h, -1, C.byref(nk), None, None, None, None, None, None)
    out = {}
    for k in range(nk.value):
        name, n, ms = C.c_char_p(), C.c_int32(0), C.c_float(0)
        w, e, b = C.c_int64(0), C.c_int64(0), C.c_int64(0)
        _check(lib.rk_fill_kernel_stats(h, k, None, C.byref(name), C.byref(n), C.byref(ms),
                                        C.byref(w), C.byref(e), C.byref(b)), "rk_fill_kernel_stats")
        out[name.value.decode()] = (int(n.value), float(ms.value), int(w.value), int(e.value), int(b.value))
    return out


class Solver:
    """A chain handle with the solve/read calls bound to it."""

    def __init__(self, chain):
        self.chain = chain
        self.L, self.K = chain.L, chain.K
        self.h = rk_chain_create(chain.L, chain.K, *chain.arrays())
        self.M = None
        if getattr(chain, "refwd", None) is not None:  # the saving sweep
            rk_chain_set_saving_sweep(self.h, chain.refwd)

    def solve(self, M: int | None = None) -> int:
        self.M = self.chain.M if M is None else int(M)
        return rk_solve(self.h, self.M)

    def solve_async(self, M, workspace_ptr, ws_bytes, stream_ptr=None) -> None:
        self.M = int(M)
        rk_solve_async(self.h, self.M, workspace_ptr, ws_bytes, stream_ptr)

    def result(self) -> int:
        return rk_result(self.h)

    def workspace_bytes(self, M: int) -> int:
        return rk_workspace_bytes(self.h, M)

    def schedule(self):
        return rk_extract_schedule(self.h)

    def set_saving_sweep(self, refwd) -> None:
        rk_chain_set_saving_sweep(self.h, refwd)

    def set_option_pruning(self, enable: bool) -> None:
        rk_set_option_pruning(self.h, enable)

    def options(self):
        """(kept [L, K] bool, k_run) under the current pruning setting."""
        return rk_chain_options(self.h, self.L, self.K)

    def row(self, s: int, t: int, want_arg: bool = True):
        return rk_read_row(self.h, s, t, self.M + 1, want_arg)

    def tradeoff_curve(self, n: int | None = None) -> np.ndarray:
        """Best schedule time at every total budget 0..n-1 (default: up to the solve's M)."""
        return rk_tradeoff_curve(self.h, self.M + 1 if n is None else n)

    def rows(self, want_arg: bool = True):
        """All rows in upper-triangle row-major order of (s,t): ([ncells, W] opt, arg)."""
        L, W = self.L, self.M + 1
        n = L * (L + 1) // 2
        opt = np.empty((n, W), dtype=np.int32)
        arg = np.empty((n, W), dtype=np.int16) if want_arg else None
        k = 0
        for s in range(L):
            for t in range(s, L):
                o, a = self.row(s, t, want_arg)
                opt[k] = o
                if want_arg:
                    arg[k] = a
                k += 1
        return opt, arg

    def fill_ms(self):
        return rk_last_fill_ms(self.h)

    def set_profiling(self, mode) -> None:
        rk_set_profiling(self.h, mode)

    def kernel_stats(self):
        return rk_fill_kernel_stats(self.h)

    def close(self) -> None:
        if self.h is not None:
            rk_chain_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
