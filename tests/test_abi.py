"""The C ABI on a host without a GPU: the library loads, exports what include/rk.h
declares, and rejects bad input before touching any device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2307_01236_amd import rk
from paper_2307_01236_amd.chaingen import make_config_chain, make_random_chain

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "rk.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rk_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = rk.load()
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(rk.EXPORTS)


def test_calibration_library_exports():
    from paper_2307_01236_amd import calib
    text = open(os.path.join(ROOT, "include", "rk_calib.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = sorted(set(re.findall(r"\b(rkc_[a-z0-9_]+)\s*\(", text)))
    assert set(names) == set(calib.EXPORTS)
    lib = calib.load()
    for n in names:
        assert hasattr(lib, n), n
    # argument checks happen before any device call
    import ctypes as C
    out = C.c_double()
    assert lib.rkc_valu_int32_rate(0, C.byref(out)) == -1
    assert lib.rkc_copy_bandwidth(17, C.byref(out)) == -1
    assert lib.rkc_copy_bandwidth(1 << 30, None) == -1
    assert lib.rkc_read_bandwidth(17, C.byref(out)) == -1
    assert lib.rkc_read_bandwidth(0, C.byref(out)) == -1
    assert lib.rkc_read_bandwidth(1 << 30, None) == -1


def test_constants_match_header():
    text = open(os.path.join(ROOT, "include", "rk.h")).read()
    for name in ("RK_OK", "RK_E_INVAL", "RK_E_OVERFLOW", "RK_E_NOMEM", "RK_E_DEVICE", "RK_E_NOT_SOLVED",
                 "RK_E_INFEASIBLE", "RK_E_BUFSZ", "RK_E_INTERNAL", "RK_FWD_NOSAVE", "RK_FWD_SAVE",
                 "RK_BWD", "RK_FREE_X"):
        m = re.search(rf"\b{name}\s*=\s*(-?\d+)", text)
        assert m and int(m.group(1)) == getattr(rk, name), name
    assert "#define RK_MAX_L 2000" in text


def test_strerror():
    assert rk.rk_strerror(0) == "ok"
    assert "invalid" in rk.rk_strerror(rk.RK_E_INVAL)
    assert rk.rk_strerror(12345) == "unknown error"


def _args(ch):
    return (ch.L, ch.K) + tuple(ch.arrays())


def _create_rc(L, K, *arrs):
    import ctypes as C
    lib = rk.load()
    h = C.c_void_p()
    arrs = [np.ascontiguousarray(a, dtype=np.int32).ravel() for a in arrs]
    ptrs = [a.ctypes.data_as(C.POINTER(C.c_int32)) for a in arrs]
    rc = lib.rk_chain_create(L, K, *ptrs, C.byref(h))
    if rc == rk.RK_OK:
        lib.rk_chain_destroy(h)
    return rc


def test_create_and_destroy_without_gpu():
    ch = make_config_chain(0)
    h = rk.rk_chain_create(*_args(ch))
    assert h.value
    rk.rk_chain_destroy(h)
    rk.rk_chain_destroy(None)


def test_create_rejects_bad_input():
    ch = make_random_chain(1, 6, 3)
    a = list(ch.arrays())
    assert _create_rc(ch.L, ch.K, *a) == rk.RK_OK
    assert _create_rc(0, ch.K, *a) == rk.RK_E_INVAL
    assert _create_rc(ch.L, 0, *a) == rk.RK_E_INVAL
    assert _create_rc(rk.RK_MAX_L + 1, ch.K, *a) == rk.RK_E_INVAL
    for j in range(len(a)):
        b = [x.copy() for x in a]
        b[j].flat[-1] = -1
        assert _create_rc(ch.L, ch.K, *b) == rk.RK_E_INVAL, j


def test_create_rejects_time_overflow():
    ch = make_random_chain(2, 8, 2)
    a = [x.copy() for x in ch.arrays()]
    # bound = L * sum_i max(fn, max_o fwd) + sum_i max_o bwd
    a[3][:] = (rk.RK_TIME_LIMIT // (8 * 8)) + 1
    assert _create_rc(ch.L, ch.K, *a) == rk.RK_E_OVERFLOW
    a[3][:] = 1
    a[1][:] = 1
    a[4][:] = 1
    a[4][0, 0] = rk.RK_TIME_LIMIT - 8 * 8 - 7
    assert _create_rc(ch.L, ch.K, *a) == rk.RK_OK
    a[4][0, 0] += 1
    assert _create_rc(ch.L, ch.K, *a) == rk.RK_E_OVERFLOW


def test_workspace_guard_for_32bit_offsets():
    # the products address an operand block with 32-bit byte offsets from its first row; the
    # widest block (a mid tile's left operands of 18 rows s) spans 18 (L - 1) rows: a chain
    # and budget whose 18 L + 64 rows span 2 GiB or more are refused rather than miscomputed
    ch = make_random_chain(3, 384, 2, xmax=7)
    h = rk.rk_chain_create(*_args(ch))
    try:
        def row_bytes(M):  # a 64-column pad (max x_i <= 7) plus the budget columns, 64-aligned
            return (64 + (M + 1 + 63) // 64 * 64) * 4
        span = 18 * ch.L + 64
        ok = max(M for M in range(70_000, 80_000, 64) if span * row_bytes(M) < 2 ** 31)
        assert rk.rk_workspace_bytes(h, ok) > 0  # ~90 GB of tables: accepted
        with pytest.raises(rk.RKError) as e:
            rk.rk_workspace_bytes(h, ok + 64)
        assert e.value.code == rk.RK_E_NOMEM
        with pytest.raises(rk.RKError) as e:
            rk.rk_workspace_bytes(h, 3_000_000)
        assert e.value.code == rk.RK_E_NOMEM
        assert rk.rk_workspace_bytes(h, 1000) > 0
    finally:
        rk.rk_chain_destroy(h)


def test_workspace_bytes():
    ch = make_config_chain(4)
    h = rk.rk_chain_create(*_args(ch))
    try:
        # three tables (Opt, the case-2 left operand and its right operand laid out at column
        # m), each with one extra all-infinity row and 32 rows of slack at either end; rows are
        # a 64-column infinity pad (max x_i = 7 here) plus the budget columns
        rows = ch.L * (ch.L + 1) // 2 + 1 + 64
        assert rk.rk_workspace_bytes(h, 6000) == 3 * rows * (64 + 6016) * 4
        assert rk.rk_workspace_bytes(h, 0) == 3 * rows * (64 + 64) * 4
        with pytest.raises(rk.RKError):
            rk.rk_workspace_bytes(h, -1)
        with pytest.raises(rk.RKError):
            rk.rk_workspace_bytes(h, rk.RK_MAX_M + 1)
    finally:
        rk.rk_chain_destroy(h)


def test_reads_before_solve_are_refused():
    ch = make_config_chain(0)
    h = rk.rk_chain_create(*_args(ch))
    try:
        for f in (lambda: rk.rk_result(h), lambda: rk.rk_extract_schedule(h),
                  lambda: rk.rk_read_row(h, 0, 0, 10), lambda: rk.rk_last_fill_ms(h)):
            with pytest.raises(rk.RKError) as e:
                f()
            assert e.value.code == rk.RK_E_NOT_SOLVED
        with pytest.raises(rk.RKError) as e:
            rk.rk_read_row(h, 3, 2, 10)
        assert e.value.code == rk.RK_E_INVAL
        with pytest.raises(rk.RKError) as e:
            rk.rk_read_row(h, 0, ch.L, 10)
        assert e.value.code == rk.RK_E_INVAL
    finally:
        rk.rk_chain_destroy(h)


def test_saving_sweep_arguments():
    """rk_chain_set_saving_sweep: negative times and too many option codes are refused,
    the time bound counts the re-forward, NULL switches the case off; the workspace of a
    solve with the case on holds H and its left operand next to Opt and ap."""
    ch = make_random_chain(3, 8, 2)
    h = rk.rk_chain_create(*_args(ch))
    try:
        W0 = rk.rk_workspace_bytes(h, 100)
        lib = rk.load()
        bad = np.zeros((ch.L, ch.K), dtype=np.int32)
        bad[2, 1] = -1
        assert lib.rk_chain_set_saving_sweep(h, bad.ctypes.data_as(C.POINTER(C.c_int32))) == rk.RK_E_INVAL
        big = np.full((ch.L, ch.K), rk.RK_TIME_LIMIT // (8 * 8) + 1, dtype=np.int32)
        assert lib.rk_chain_set_saving_sweep(h, big.ctypes.data_as(C.POINTER(C.c_int32))) == rk.RK_E_OVERFLOW
        assert rk.rk_workspace_bytes(h, 100) == W0  # unchanged after the refusals
        ok = np.ones((ch.L, ch.K), dtype=np.int32)
        rk.rk_chain_set_saving_sweep(h, ok)
        assert 3 * rk.rk_workspace_bytes(h, 100) == 5 * W0  # two more tables of the same shape
        rk.rk_chain_set_saving_sweep(h, None)
        assert rk.rk_workspace_bytes(h, 100) == W0
        assert lib.rk_chain_set_saving_sweep(None, None) == rk.RK_E_INVAL
    finally:
        rk.rk_chain_destroy(h)
    # codes up to L + 2K - 1 must fit int16
    K = 16384  # L + K fits, L + 2K does not
    wide = make_random_chain(4, 1, K)
    h = rk.rk_chain_create(*_args(wide))
    try:
        ok = np.zeros((1, K), dtype=np.int32)
        assert rk.load().rk_chain_set_saving_sweep(h, ok.ctypes.data_as(C.POINTER(C.c_int32))) == rk.RK_E_INVAL
    finally:
        rk.rk_chain_destroy(h)


def test_profiling_modes():
    """rk_set_profiling takes 0 (off), 1 (timing) and 2 (timing and device counts); other
    modes and a NULL handle are refused."""
    ch = make_config_chain(0)
    h = rk.rk_chain_create(*_args(ch))
    lib = rk.load()
    try:
        for mode in (1, 2, 0):
            assert lib.rk_set_profiling(h, mode) == rk.RK_OK
        for mode in (-1, 3):
            assert lib.rk_set_profiling(h, mode) == rk.RK_E_INVAL
        assert lib.rk_set_profiling(None, 1) == rk.RK_E_INVAL
    finally:
        rk.rk_chain_destroy(h)
