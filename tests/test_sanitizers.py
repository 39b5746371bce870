"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

- The CPU oracle (oracle/rko.c) built with both sanitizers runs on chains of every kind
  the pins use (ties, zeros, the saving sweep, the benchmark's smallest workloads) and must
  report exactly what the normal build reports.
- The solver library's host precompute (csrc/rk_host.cpp: derived quantities, the
  dominance test, the store-everything budgets, the option slots) built with both
  sanitizers runs over 400 generated chains, valid and invalid.
Any sanitizer report aborts the driver (-fno-sanitize-recover), which fails the test.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from paper_2307_01236_amd.chaingen import make_config_chain, make_random_chain, with_refwd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")


def _have(tool):
    return shutil.which(tool) is not None


def _chains():
    out = [make_config_chain(0), make_config_chain(1)]
    for seed in range(12):
        ch = make_random_chain(880 + seed, 1 + seed % 9, 1 + seed % 4, allow_zero=seed % 3 == 0,
                               small_times=seed % 2 == 0, uniform=seed % 5 == 4)
        out.append(with_refwd(ch, seed) if seed % 2 else ch)
    return out


def _write(chains, path):
    with open(path, "wb") as f:
        for ch in chains:
            rf = getattr(ch, "refwd", None)
            np.array([ch.L, ch.K, ch.M, rf is not None], dtype=np.int32).tofile(f)
            for a in ch.arrays():
                np.ascontiguousarray(a, dtype=np.int32).tofile(f)
            if rf is not None:
                np.ascontiguousarray(rf, dtype=np.int32).tofile(f)


def _expected(ch):
    sol = oracle.solve(ch)
    opt = sol.opt.astype(np.int64)
    osum = int(opt[opt != oracle.INF].sum())
    asum = int(sol.arg.astype(np.int64).sum())
    mf = oracle.min_feasible(ch)
    mfs = int(mf[mf <= 1_000_000_000].sum())
    if sol.answer == oracle.INF:
        return f"{sol.answer} {osum} {asum} 0 -1 -1 {mfs}"
    ops, _ = oracle.schedule(sol)
    ok, tm, pk, _ = oracle.simulate(ch, ops)
    assert ok
    return f"{sol.answer} {osum} {asum} {len(ops)} {tm} {pk} {mfs}"


@pytest.mark.skipif(not _have("gcc"), reason="gcc is needed")
def test_oracle_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_san"
    subprocess.check_call(["gcc", "-std=c11", *SAN, "-I", os.path.join(ROOT, "oracle"),
                           os.path.join(ROOT, "oracle", "rko.c"), os.path.join(HERE, "oracle_driver.c"),
                           "-o", str(exe)])
    chains = _chains()
    data = tmp_path / "chains.bin"
    _write(chains, data)
    res = subprocess.run([str(exe), str(data)], capture_output=True, text=True, env=ENV, timeout=300)
    assert res.returncode == 0, res.stderr[-4000:]
    got = res.stdout.strip().splitlines()
    assert got == [_expected(ch) for ch in chains]


@pytest.mark.skipif(not _have("g++"), reason="g++ is needed")
def test_host_precompute_under_sanitizers(tmp_path):
    exe = tmp_path / "host_san"
    csrc = os.path.join(ROOT, "paper_2307_01236_amd", "csrc")
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"), "-I", csrc,
                           os.path.join(csrc, "rk_host.cpp"), os.path.join(HERE, "host_driver.cpp"),
                           "-o", str(exe)])
    res = subprocess.run([str(exe)], capture_output=True, text=True, env=ENV, timeout=300)
    assert res.returncode == 0, (res.stdout[-2000:], res.stderr[-4000:])
    lines = res.stdout.strip().splitlines()
    assert len(lines) == 400
    assert sum(" ok " in ln for ln in lines) > 250 and any(" rc -2" in ln for ln in lines)
