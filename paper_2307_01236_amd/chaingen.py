"""Seeded synthetic block chains for the rk-Rotor solver.

This module only draws inputs.  It holds none of the solver's arithmetic: no
derived quantity of the dynamic program (saved sizes, validity thresholds,
prefix sums, table values) is computed here.  Both the HIP path and the CPU
oracle receive the arrays it returns.

A chain is what rk-Rotor takes as input (Alg. 1, the ``sols`` argument, and
the notation of App. C): L blocks, each with a no-save forward F^0
(time, temporary memory) and K saving options o, each option with a forward
time r(F^o), a backward time r(B^o), the size of the intermediates it keeps
until its backward, and temporary memory for its forward and backward.
Activation sizes x_0..x_L (x_L is the chain output) complete it.

The five named workloads follow the cost recipe of the benchmark
configurations: per block, forward time f ~ U[100,1000], backward base 2f,
saved-activation size a ~ U[2, 2M/L], input-checkpoint size x ~ U[1, M/(2L)];
option k of K keeps floor(a (K-k)/K) slots, its backward costs
2f + floor(f k ub / (K-1)) with ub ~ U(0.8,1), and its peak overhead is
ceil(a up) with up ~ U(0.2,0.6).  They stand in for the measured GPT2,
ResNet and RegNet chains of the paper's experiments (Sec. 4), which are not
available.
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np

__all__ = ["Chain", "CONFIGS", "make_config_chain", "make_random_chain", "make_grid_chain",
           "config_by_name", "with_refwd"]


@dataclasses.dataclass
class Chain:
    """Inputs of one rk-Rotor solve, as contiguous int32 arrays.

    x        [L+1]  activation sizes x_0..x_L
    fn_time  [L]    r(F_i^0), the no-save forward
    fn_tmp   [L]    tmp(F_i^0)
    fwd, bwd [L,K]  r(F_i^o), r(B_i^o)
    mem      [L,K]  size of the intermediates option o keeps for its backward
    tmp_fwd, tmp_bwd [L,K]  tmp(F_i^o), tmp(B_i^o)
    M        budget (memory slots) the workload is solved at
    refwd    [L,K]  or None: time to compute x_{i+1} again from the intermediates F_i^o
             kept (the saving sweep of the paper's sub-optimality remark (ii), Sec. 3.4);
             None leaves it out
    """

    L: int
    K: int
    x: np.ndarray
    fn_time: np.ndarray
    fn_tmp: np.ndarray
    fwd: np.ndarray
    bwd: np.ndarray
    mem: np.ndarray
    tmp_fwd: np.ndarray
    tmp_bwd: np.ndarray
    M: int
    name: str = "chain"
    refwd: np.ndarray | None = None

    def arrays(self):
        return (self.x, self.fn_time, self.fn_tmp, self.fwd, self.bwd, self.mem,
                self.tmp_fwd, self.tmp_bwd)

    def sha256(self) -> str:
        h = hashlib.sha256()
        h.update(np.array([self.L, self.K, self.M], dtype=np.int64).tobytes())
        for a in self.arrays():
            h.update(np.ascontiguousarray(a, dtype=np.int32).tobytes())
        if self.refwd is not None:
            h.update(b"refwd")
            h.update(np.ascontiguousarray(self.refwd, dtype=np.int32).tobytes())
        return h.hexdigest()

    def sub(self, s: int, t: int) -> "Chain":
        """Blocks s..t (inclusive) as a chain of their own (same M)."""
        return Chain(L=t - s + 1, K=self.K, x=self.x[s:t + 2].copy(),
                     fn_time=self.fn_time[s:t + 1].copy(), fn_tmp=self.fn_tmp[s:t + 1].copy(),
                     fwd=self.fwd[s:t + 1].copy(), bwd=self.bwd[s:t + 1].copy(),
                     mem=self.mem[s:t + 1].copy(), tmp_fwd=self.tmp_fwd[s:t + 1].copy(),
                     tmp_bwd=self.tmp_bwd[s:t + 1].copy(), M=self.M,
                     name=f"{self.name}[{s}:{t}]",
                     refwd=None if self.refwd is None else self.refwd[s:t + 1].copy())

    def options(self, keep) -> "Chain":
        """The same blocks with only the saving options listed in `keep` (in that order).
        keep=[0] leaves each block the option that keeps all its intermediates, which is
        Rotor's choice set (store everything or nothing per block)."""
        keep = list(keep)
        pick = lambda a: np.ascontiguousarray(a[:, keep])
        return Chain(L=self.L, K=len(keep), x=self.x.copy(), fn_time=self.fn_time.copy(),
                     fn_tmp=self.fn_tmp.copy(), fwd=pick(self.fwd), bwd=pick(self.bwd),
                     mem=pick(self.mem), tmp_fwd=pick(self.tmp_fwd), tmp_bwd=pick(self.tmp_bwd),
                     M=self.M, name=f"{self.name}{{options {keep}}}",
                     refwd=None if self.refwd is None else pick(self.refwd))

# name, L, K, M, block-structure kind
CONFIGS = [
    dict(name="chain_L8_K3_M500", L=8, K=3, M=500, kind="hetero"),
    dict(name="gpt_like_L64_K5_M1000", L=64, K=5, M=1000, kind="uniform"),
    dict(name="resnet_like_L128_K8_M2000", L=128, K=8, M=2000, kind="hetero"),
    dict(name="regnet_like_L256_K8_M4000", L=256, K=8, M=4000, kind="downsample4"),
    dict(name="deep_gpt_like_L384_K16_M6000", L=384, K=16, M=6000, kind="uniform"),
]


def config_by_name(name: str) -> int:
    for i, c in enumerate(CONFIGS):
        if c["name"] == name:
            return i
    raise KeyError(name)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64).astype(np.int32))


def _options(f, a, ub, up, K):
    """Per-option costs of the benchmark recipe (input synthesis only)."""
    L = len(f)
    k = np.arange(K)
    fwd = np.repeat(f[:, None], K, axis=1)
    if K > 1:
        extra = np.floor(f[:, None].astype(np.float64) * k[None, :] * ub / (K - 1)).astype(np.int64)
    else:
        extra = np.zeros((L, 1), dtype=np.int64)
    bwd = 2 * f[:, None] + extra
    mem = (a[:, None] * (K - k[None, :])) // K
    tmp = np.ceil(a[:, None].astype(np.float64) * up).astype(np.int64)
    return fwd, bwd, mem, tmp


def make_config_chain(cfg: int | str, rep: int = 0) -> Chain:
    """The seeded chain of a benchmark configuration (seed = 1000*cfg + rep)."""
    if isinstance(cfg, str):
        cfg = config_by_name(cfg)
    c = CONFIGS[cfg]
    L, K, M, kind = c["L"], c["K"], c["M"], c["kind"]
    rng = np.random.Generator(np.random.PCG64(1000 * cfg + rep))
    xmax = M // (2 * L)
    amax = (2 * M) // L
    x = rng.integers(1, xmax, size=L + 1, endpoint=True)
    f = rng.integers(100, 1000, size=L, endpoint=True)
    a = rng.integers(2, amax, size=L, endpoint=True)
    ub = rng.uniform(0.8, 1.0, size=(L, K))
    up = rng.uniform(0.2, 0.6, size=(L, K))
    if kind == "downsample4":
        sel = (np.arange(L) % 4) == 3
        a = np.where(sel, 4 * a, a)
        f = np.where(sel, 2 * f, f)
    elif kind == "uniform":
        x = np.full(L + 1, x[0])
        a = np.full(L, a[0])
        ub = np.repeat(ub[:1], L, axis=0)
        up = np.repeat(up[:1], L, axis=0)
        jit = rng.uniform(0.9, 1.1, size=L)
        f = np.array([int(round(f[0] * j)) for j in jit], dtype=np.int64)
    fwd, bwd, mem, tmp = _options(f, a, ub, up, K)
    return Chain(L=L, K=K, x=_i32(x), fn_time=_i32(f), fn_tmp=_i32(tmp.min(axis=1)),
                 fwd=_i32(fwd), bwd=_i32(bwd), mem=_i32(mem), tmp_fwd=_i32(tmp),
                 tmp_bwd=_i32(tmp), M=M, name=c["name"])


def make_random_chain(seed: int, L: int, K: int, *, M: int | None = None, xmax: int = 8,
                      amax: int = 12, tmax: int = 6, tmin: int = 1, allow_zero: bool = False,
                      uniform: bool = False, small_times: bool = False,
                      independent_tmp: bool = True) -> Chain:
    """Fuzz chain with free per-option parameters.

    allow_zero  sizes and temporaries may be 0
    uniform     every block copies block 0 (tie-heavy)
    small_times times drawn from a handful of values (more ties)
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    lo = 0 if allow_zero else 1
    tlo = 1
    thi = 1000 if not small_times else 4

    def draw_block():
        fn_t = int(rng.integers(0 if allow_zero else tlo, thi, endpoint=True))
        fn_m = int(rng.integers(0 if allow_zero else tmin, tmax, endpoint=True))
        fw = rng.integers(0 if allow_zero else tlo, thi, size=K, endpoint=True)
        bw = rng.integers(0 if allow_zero else tlo, 2 * thi, size=K, endpoint=True)
        me = rng.integers(lo, amax, size=K, endpoint=True)
        tf = rng.integers(0 if allow_zero else tmin, tmax, size=K, endpoint=True)
        tb = rng.integers(0 if allow_zero else tmin, tmax, size=K, endpoint=True) if independent_tmp else tf
        return fn_t, fn_m, fw, bw, me, tf, tb

    blocks = [draw_block() for _ in range(1 if uniform else L)]
    if uniform:
        blocks = blocks * L
    x = rng.integers(lo, xmax, size=L + 1, endpoint=True)
    if uniform:
        x = np.full(L + 1, x[0])
    fn_time = _i32([b[0] for b in blocks])
    fn_tmp = _i32([b[1] for b in blocks])
    fwd = _i32(np.stack([b[2] for b in blocks]))
    bwd = _i32(np.stack([b[3] for b in blocks]))
    mem = _i32(np.stack([b[4] for b in blocks]))
    tf = _i32(np.stack([b[5] for b in blocks]))
    tb = _i32(np.stack([b[6] for b in blocks]))
    if M is None:
        # a little above what storing everything would need
        M = int(x.sum() + mem.max(axis=1).sum() + tf.max() + tb.max() + 2)
    return Chain(L=L, K=K, x=_i32(x), fn_time=fn_time, fn_tmp=fn_tmp, fwd=fwd, bwd=bwd,
                 mem=mem, tmp_fwd=tf, tmp_bwd=tb, M=int(M), name=f"random{seed}_L{L}_K{K}")


def with_refwd(ch: Chain, seed: int, lo: float = 0.0, hi: float = 1.0) -> Chain:
    """The same chain with re-forward times for the saving sweep: recomputing x_{i+1} from
    the intermediates option o kept costs floor(r(F_i^0) * U[lo, hi]) (input synthesis
    only; hi <= 1 keeps it below a full forward)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    u = rng.uniform(lo, hi, size=(ch.L, ch.K))
    refwd = np.floor(ch.fn_time.astype(np.float64)[:, None] * u).astype(np.int64)
    return dataclasses.replace(ch, refwd=_i32(refwd), name=f"{ch.name}+refwd{seed}")


def _grid_options(rng, n_peak: int, n_save: int):
    """Per-option costs of one block type from an emulated option search on a budget grid.

    Stand-in for the paper's block-level solver (Sec. 3, Phase 2), which is not part of this
    build: a block produces n tensors, tensor j of size sz_j costing rc_j to compute; a few
    are cheap to recompute and large (dropout/gelu-like), the rest costly.  A block schedule
    keeps a subset S of them from the forward to the backward and recomputes the others
    there.  For each pair (M_peak, M_save) of the grid (M_peak evenly spaced between the
    peaks of keeping nothing and keeping everything, M_save evenly spaced in [0, M_peak]),
    the subset with the least recomputation whose kept size fits M_save and whose backward
    peak (kept size + the largest recomputed tensor + a workspace) fits M_peak is taken, by
    enumeration.  Options come in grid order; different pairs often give the same subset.
    """
    n = int(rng.integers(6, 11))
    cheap = rng.random(n) < 0.35
    sz = np.where(cheap, rng.integers(8, 25, size=n), rng.integers(2, 12, size=n))
    rc = np.where(cheap, rng.integers(1, 6, size=n), rng.integers(40, 250, size=n))
    work = int(rng.integers(1, 6))
    masks = np.arange(1 << n)
    bits = (masks[:, None] >> np.arange(n)[None, :]) & 1
    kept_size = bits @ sz
    recompute = (1 - bits) @ rc
    tmp_b = work + np.where(bits.all(axis=1), 0, ((1 - bits) * sz[None, :]).max(axis=1))
    peak = kept_size + tmp_b
    f = int(rc.sum())
    lo, hi = int(peak[0]), int(peak[-1])
    opts = []
    for mp in np.linspace(lo, max(lo, hi), n_peak):
        for ms in np.linspace(0, mp, n_save):
            ok = (kept_size <= ms) & (peak <= mp)
            ok[0] = True  # keeping nothing always fits: M_peak >= its peak
            key = np.where(ok, recompute, np.iinfo(np.int64).max)
            best = np.flatnonzero(key == key.min())
            j = best[np.argmin(kept_size[best])]
            opts.append((f, 2 * f + int(recompute[j]), int(kept_size[j]), work, int(tmp_b[j])))
    return f, work, np.array(opts, dtype=np.int64)


def make_grid_chain(seed: int, L: int, n_peak: int = 20, n_save: int = 20, *, types: int = 2,
                    M: int | None = None, xmax: int = 6) -> Chain:
    """A chain of `types` block types repeated in turn (GPT-like: attention and MLP blocks),
    each with the n_peak * n_save options of an emulated grid search (see _grid_options);
    identical blocks share their options, as in the paper.  Many options are repeats."""
    rng = np.random.Generator(np.random.PCG64(seed))
    tys = [_grid_options(rng, n_peak, n_save) for _ in range(types)]
    x = rng.integers(1, xmax, size=L + 1, endpoint=True)
    K = n_peak * n_save
    fwd, bwd, mem, tf, tb = (np.empty((L, K), dtype=np.int64) for _ in range(5))
    fn_time, fn_tmp = np.empty(L, dtype=np.int64), np.empty(L, dtype=np.int64)
    for i in range(L):
        f, work, o = tys[i % types]
        fwd[i], bwd[i], mem[i], tf[i], tb[i] = o.T
        fn_time[i], fn_tmp[i] = f, work
    if M is None:
        M = int((x.sum() + mem.max(axis=1).sum()) // 3)
    return Chain(L=L, K=K, x=_i32(x), fn_time=_i32(fn_time), fn_tmp=_i32(fn_tmp), fwd=_i32(fwd),
                 bwd=_i32(bwd), mem=_i32(mem), tmp_fwd=_i32(tf), tmp_bwd=_i32(tb), M=M,
                 name=f"grid_L{L}_K{K}_s{seed}")


def store_all_bound(ch: Chain) -> int:
    """A budget at which every activation and every option's data fits at once.

    Used only to pick test budgets "above store-all"; a generous over-estimate.
    """
    return int(ch.x.sum() + ch.mem.max(axis=1).sum() + ch.tmp_fwd.max() + ch.tmp_bwd.max()
               + ch.fn_tmp.max() + 1)


def relaxations(L: int, K: int, M: int) -> int:
    """Candidate evaluations of one fill: (M+1) * sum_d (L-d)(K+d)."""
    return (M + 1) * (K * L * (L + 1) // 2 + (L ** 3 - L) // 6)


def cells(L: int, M: int) -> int:
    return (M + 1) * L * (L + 1) // 2


if __name__ == "__main__":  # pragma: no cover
    for i, c in enumerate(CONFIGS):
        ch = make_config_chain(i)
        print(i, c["name"], ch.sha256()[:16], "x", ch.x[:4], "f", ch.fn_time[:4],
              "mem", ch.mem[0], "tmp", ch.tmp_fwd[0], "bwd", ch.bwd[0],
              f"relax={relaxations(ch.L, ch.K, ch.M):.3e}")
