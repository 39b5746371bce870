"""Benchmark of the rk-Rotor solve on one MI355X.

One step is one pass of the whole hot path over one chain: the table fill for
every span and every budget (App. C, Alg. 2), the answer read-back, and the
schedule (Alg. 3) copied to the host.  The chain is the deep transformer-like
workload, 384 blocks with 16 options each at a 6000-slot budget, created and
uploaded before the timed region; the table lives in a torch allocation and
the solve runs on a torch stream.

Prints one JSON line on stdout.  ``value`` is DP relaxations per second of
the whole step (relaxations = candidate evaluations of the recurrence,
(M+1) * sum_d (L-d)(K+d)).  ``roofline`` reports the dominant fill kernel (the
kind with the most device time, from HIP events the runtime records with each
dispatch on the solve's stream) against the roof that binds it: HBM bandwidth for its compulsory table
traffic (every row a launch reads counted once, plus the rows it writes) or the
VALU integer peak for its relaxations (an add and a min each), whichever
fraction is higher, both counting only what the kernels evaluate (a profiled step
with the counting kernel variants reports the candidates and rows that the lower
bound lets them skip); the other one is reported beside it; both are also priced
against what this GPU sustains (``measured_ceilings``: int32 add/min chains over
the whole chip, a 1 GiB device copy and a 1 GiB device read; a kernel's bandwidth ceiling
is the time-weighted mix of the read rate and the write rate the copy implies, for its own
share of bytes written).  ``cpu_baseline``
times the CPU oracle (one core) on a bounded part of the same chain.  After
the timed and profiled steps, ``tradeoff`` and ``option_pruning`` report the
memory/time trade-off curve of the fill against Rotor's (Sec. 4) and the effect
of option pruning on a chain with an emulated budget-grid option search, and
``other_workloads`` the fill times of the four smaller workloads (``--extras 0``
skips all three, for profiler runs that should see one workload).
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "DP relaxations/sec + wall solve time per chain on 1 MI355X; % HBM/VALU roofline"
WORKLOAD_CFG = 4
# MI355X: 256 CUs x 4 SIMD16 = 64 int32 lanes per CU per clock at 2.4 GHz
VALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
OPS_PER_RELAX = 2  # one add and one min per candidate
HBM_PEAK_GBS = 8000.0


def write_bytes_per_fill(kernel: str, L: int, W: int):
    """Bytes of a fill kernel's compulsory traffic that are writes, per fill (None if not
    tabulated).  The finalize writes the Opt row of every span and the ap row of every span
    that does not end at block L-1; the band product writes one partial row per span of
    each 32-span band."""
    row = W * 4
    if kernel == "k_finalize":
        return L * L * row
    if kernel == "k_product":
        return sum(L - dd for tau in range(32, L, 32) for dd in range(tau, min(tau + 32, L))) * row
    return None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary,
    if it was taken on the kernel source as it is now; else (None, None)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.json")
    if not os.path.exists(path):
        return None, None
    with open(path) as f:
        prof = json.load(f)
    with open(os.path.join(ROOT, prof["kernels_source"]), "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    k = prof["kernels"].get(kernel)
    if sha != prof["kernels_source_sha256"] or k is None:
        return None, None
    return k["hbm_bytes_per_dispatch"], None


def cpu_baseline(ch, nblocks: int):
    import oracle
    from paper_2307_01236_amd.chaingen import relaxations
    if not os.path.exists(oracle.LIB):
        oracle.build(force=False)
    sub = ch.sub(0, nblocks - 1)
    t0 = time.perf_counter()
    oracle.solve(sub)
    dt = time.perf_counter() - t0
    r = relaxations(sub.L, sub.K, sub.M)
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), model)
    except OSError:
        pass
    return {"value": r / dt, "unit": "relaxations/s", "cores": 1, "kind": "oracle",
            "sample": f"blocks 0..{nblocks - 1} of the same chain, M={sub.M}: {r:.3e} relaxations "
                      f"in {dt:.2f} s on one host core",
            "seconds": dt, "cpu_model": model, "host_cpus": os.cpu_count()}


def extras(ch, s, M, oracle_rate=None):
    """Reports beside the benchmark: the trade-off curve against Rotor's, option pruning, the
    smaller workloads and the saving sweep."""
    from paper_2307_01236_amd import rk
    from paper_2307_01236_amd.chaingen import make_grid_chain, relaxations

    # Sec. 4's comparison with Rotor on the same chain: the trade-off curve of this fill (every
    # budget's optimum) against one of Rotor's choice set (keep everything or nothing per
    # block: option 0), as overhead over the time with no recomputation
    t = time.perf_counter()
    curve = s.tradeoff_curve()
    curve_ms = (time.perf_counter() - t) * 1e3
    rot = rk.Solver(ch.options([0]))
    rot.solve(M)
    rcurve = rot.tradeoff_curve()
    rot.close()
    ideal = int((ch.fwd.astype("int64") + ch.bwd).min(axis=1).sum())
    budgets = [int(M * f) for f in (0.1, 0.2, 0.3, 0.5, 0.75, 1.0)]
    ovh = lambda v: None if v == rk.RK_INF else round(int(v) / ideal - 1.0, 4)
    tradeoff = {"curve_read_ms": curve_ms, "budgets": budgets,
                "rk_rotor_overhead": [ovh(curve[b]) for b in budgets],
                "rotor_overhead": [ovh(rcurve[b]) for b in budgets],
                "min_budget_rk_rotor": int((curve < rk.RK_INF).argmax()),
                "min_budget_rotor": int((rcurve < rk.RK_INF).argmax())}
    log(f"trade-off: {tradeoff}")

    # Option pruning (Sec. 3, Phase 2: the budget grid of the option search repeats options):
    # an emulated 20 x 20 grid search gives 400 options per block on a 96-block chain; the
    # fill with the distinct ones only against the fill with all of them
    g = make_grid_chain(1, 96)
    pruning = {"workload": g.name, "L": g.L, "K": g.K, "M": g.M}
    gs = rk.Solver(g)
    for on in (True, False):
        gs.set_option_pruning(on)
        k_run = gs.options()[1]
        fills = []
        for _ in range(4):
            gs.solve(g.M)
            fills.append(gs.fill_ms()[0])
        key = "pruned" if on else "all_options"
        pruning[key] = {"k_run": k_run, "fill_ms": statistics.median(fills[1:]),
                        "relaxations": relaxations(g.L, k_run, g.M), "answer": gs.result()}
    gs.close()
    log(f"option pruning: {pruning}")

    # the smaller workloads: fill time (captured launch sequence replayed, median of 5 after
    # one warm-up), launches and relaxations per second (launch latency bounds the small
    # ones); the wall time of a synchronous solve (fill + answer) and of the schedule; the
    # oracle's time for the whole chain on one host core where it takes seconds, else
    # extrapolated from the oracle's measured rate on the benchmark sample
    import oracle
    from paper_2307_01236_amd.chaingen import CONFIGS, make_config_chain
    others = []
    for cfg in range(len(CONFIGS)):
        c = make_config_chain(cfg)
        if c.name == ch.name:
            continue
        cs = rk.Solver(c)
        fills, walls = [], []
        for _ in range(6):
            t = time.perf_counter()
            cs.solve(c.M)
            walls.append((time.perf_counter() - t) * 1e3)
            fills.append(cs.fill_ms()[0])
        t = time.perf_counter()
        cs.schedule()
        sched = (time.perf_counter() - t) * 1e3
        ms = statistics.median(fills[1:])
        r = relaxations(c.L, c.K, c.M)
        row = {"workload": c.name, "launches": cs.fill_ms()[1], "fill_ms": ms, "relaxations_per_s": r / (ms * 1e-3),
               "wall_solve_ms": statistics.median(walls[1:]), "schedule_ms": sched}
        cs.close()
        if r <= 2e9 or oracle_rate is None:
            t = time.perf_counter()
            oracle.solve(c)
            row["oracle_s"] = time.perf_counter() - t
            row["oracle_kind"] = "measured, whole chain, one host core"
        else:
            row["oracle_s"] = r / oracle_rate
            row["oracle_kind"] = "extrapolated from the benchmark sample's rate, one host core"
        others.append(row)
    log(f"other workloads: {others}")

    # the saving sweep (the third case of the recurrence) on the benchmark chain: re-forward
    # times drawn up to half a no-save forward; the fill carries the H tables beside Opt
    from paper_2307_01236_amd.chaingen import with_refwd
    sw = with_refwd(ch, 1, 0.0, 0.5)
    ss = rk.Solver(sw)
    fills = []
    for _ in range(4):
        ss.solve(M)
        fills.append(ss.fill_ms()[0])
    sweep = {"workload": sw.name, "M": M, "fill_ms": statistics.median(fills[1:]), "launches": ss.fill_ms()[1],
             "answer": ss.result(), "answer_without": int(s.result()),
             "schedule_refwd_ops": int((ss.schedule()[0][:, 0] == rk.RK_REFWD).sum())}
    ss.close()
    log(f"saving sweep: {sweep}")

    return tradeoff, pruning, others, sweep


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=WORKLOAD_CFG)
    ap.add_argument("--cpu-blocks", type=int, default=144, help="oracle sample size (0: skip)")
    ap.add_argument("--extras", type=int, default=1,
                    help="0: skip the trade-off, option-pruning and other-workload reports")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized buffer 3 times (to scale HBM byte counters) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 3}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the solver runs on a single MI355X and this build "
              f"has no multi-GPU path (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2307_01236_amd import rk
    from paper_2307_01236_amd.chaingen import CONFIGS, cells, make_config_chain, relaxations

    torch.cuda.set_device(0)
    ch = make_config_chain(args.config)
    M = ch.M
    relax = relaxations(ch.L, ch.K, M)
    ncells = cells(ch.L, M)
    log(f"workload {ch.name}: L={ch.L} K={ch.K} M={M} relaxations={relax:.3e} sha={ch.sha256()[:16]}")

    # cold solves (synchronous rk_solve on a fresh chain handle: upload, table allocation,
    # capture of the launch sequence, fill).  The first one in the process also pays for the
    # runtime loading the library's kernels; the second is what a new chain costs after that.
    cold_ms = {}
    for key in ("first_in_process", "new_chain_handle"):
        t = time.perf_counter()
        cold = rk.Solver(ch)
        cold.solve(M)
        cold_ms[key] = (time.perf_counter() - t) * 1e3
        cold.close()

    s = rk.Solver(ch)
    nbytes = s.workspace_bytes(M)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    stream = torch.cuda.Stream()

    def step():
        s.solve_async(M, ws.data_ptr(), nbytes, stream.cuda_stream)
        ans = s.result()
        ops, _ = s.schedule()
        return ans, len(ops)

    for i in range(args.warmup):
        ans, nops = step()
        log(f"warmup {i}: answer={ans} ops={nops}")

    # timed steps: the production path (the fill replays its captured launch sequence);
    # HIP events around each fill on the solve's stream give the device fill time
    fill_ms = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ans, nops = step()
        fill_ms.append(s.fill_ms()[0])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step, fill median {statistics.median(fill_ms):.3f} ms")

    # the same steps again with the kernels launched one by one, each dispatch recording a
    # pair of HIP events at the kernel's start and end: per-kernel durations for the roofline
    s.set_profiling(1)
    kern = {}
    for i in range(args.steps):
        step()
        for name, (n, ms, work, _, _) in s.kernel_stats().items():
            a = kern.setdefault(name, [0, 0.0, 0, 0, 0])
            a[0] += n
            a[1] += ms
            a[2] += work
    # one more step with the counting variants of the kernels (slower, not timed): the
    # candidates each kind evaluates and the table rows they read, net of what the lower
    # bound lb(s,t) + P(s,i) skips (the same in every step, up to the mid tiles whose
    # bound test races with the folds of their launch's other tiles)
    s.set_profiling(2)
    step()
    for name, (_, _, _, evaluated, moved) in s.kernel_stats().items():
        kern[name][3] = evaluated * args.steps
        kern[name][4] = moved * args.steps
    s.set_profiling(0)

    # solve wall time without the schedule, warm (synchronous rk_solve on the library's table)
    wall = []
    for _ in range(3):
        t = time.perf_counter()
        s.solve(M)
        wall.append((time.perf_counter() - t) * 1e3)
    t = time.perf_counter()
    s.schedule()
    sched_ms = (time.perf_counter() - t) * 1e3

    cpu = None
    if args.cpu_blocks > 0:
        log(f"cpu baseline: oracle on {args.cpu_blocks} blocks ...")
        cpu = cpu_baseline(ch, min(args.cpu_blocks, ch.L))
        cpu["whole_chain_s_extrapolated"] = relax / cpu["value"]
        log(f"cpu baseline: {cpu['value']:.3e} relax/s ({cpu['seconds']:.1f} s)")

    tradeoff = pruning = others = sweep = None
    if args.extras:  # other chains' fills: after the timed and profiled steps
        tradeoff, pruning, others, sweep = extras(ch, s, M, cpu["value"] if cpu else None)

    # dominant kernel: the one with the most device time; both of its roofs per launch
    dname, (dn, dms, _, dwork, dbytes) = max(kern.items(), key=lambda kv: kv[1][1])
    per_launch_s = dms / dn * 1e-3
    ops_per_launch = OPS_PER_RELAX * dwork / dn
    bytes_per_launch = dbytes / dn
    valu = {"bound": "alu", "achieved": ops_per_launch / per_launch_s / 1e12, "peak": VALU_PEAK_TOPS,
            "unit": "TOP/s", "work_per_launch": ops_per_launch}
    valu["frac"] = valu["achieved"] / VALU_PEAK_TOPS
    hbm = {"bound": "hbm", "achieved": bytes_per_launch / per_launch_s / 1e9, "peak": HBM_PEAK_GBS,
           "unit": "GB/s", "work_per_launch": bytes_per_launch}
    hbm["frac"] = hbm["achieved"] / HBM_PEAK_GBS
    bind, other = (hbm, valu) if hbm["frac"] >= valu["frac"] else (valu, hbm)
    traffic, _ = measured_traffic(ch.name, dname)
    roofline = dict(bind)
    roofline.update({
        "traffic": traffic, "kernel": dname, "launches_per_step": dn / args.steps,
        "avg_launch_ms": dms / dn, "other_roof": other,
        "basis": "relaxations the kernel evaluates and table rows it reads: candidates of cells past "
                 "the budget from which storing everything fits are written in closed form, and those "
                 "that the lower bound lb(s,t) + P(s,i) rules out are skipped (counted on the device)",
    })
    # the whole fill against both roofs: every relaxation of the recurrence (nominal) and the
    # ones the kernels evaluate, and the compulsory table traffic of all launches
    fill_s = statistics.median(fill_ms) * 1e-3
    evaluated = sum(v[3] for v in kern.values()) / args.steps
    table_bytes = sum(v[4] for v in kern.values()) / args.steps
    # every fill kernel against both roofs (per launch, from the same profiled steps), with
    # its measured HBM traffic per launch where the committed counter summary is current
    roofline["per_kernel"] = {}
    for name, (n, ms, _, work, moved) in kern.items():
        if n == 0 or ms <= 0 or work == 0:
            continue
        t_s = ms / n * 1e-3
        meas, _ = measured_traffic(ch.name, name)
        roofline["per_kernel"][name] = {
            "launches_per_step": n / args.steps, "avg_launch_ms": ms / n,
            "valu_frac": OPS_PER_RELAX * work / n / t_s / 1e12 / VALU_PEAK_TOPS,
            "hbm_frac_compulsory": moved / n / t_s / 1e9 / HBM_PEAK_GBS,
            "measured_bytes_per_launch": meas,
            "hbm_frac_measured": meas / t_s / 1e9 / HBM_PEAK_GBS if meas is not None else None,
        }
    roofline["whole_fill"] = {
        "fill_ms": fill_s * 1e3, "launches": sum(v[0] for v in kern.values()) / args.steps,
        "relaxations_nominal": relax, "relaxations_evaluated": evaluated,
        "valu_frac_nominal": OPS_PER_RELAX * relax / fill_s / 1e12 / VALU_PEAK_TOPS,
        "valu_frac_evaluated": OPS_PER_RELAX * evaluated / fill_s / 1e12 / VALU_PEAK_TOPS,
        "table_bytes": table_bytes, "hbm_frac_compulsory": table_bytes / fill_s / 1e9 / HBM_PEAK_GBS,
    }

    # what this GPU sustains, next to the published peaks: int32 add+min chains over the
    # whole chip, a 1 GiB device copy (bytes read plus written) and a 1 GiB device read.
    # A copy's time is taken as its read time plus its write time, which gives the write
    # rate; a kernel's bandwidth ceiling is then its bytes over the time its reads and
    # writes would take at those rates.
    from paper_2307_01236_amd import calib
    measured = {"valu_int32_tops": calib.valu_int32_rate() / 1e12,
                "copy_gbs": calib.copy_bandwidth(1 << 30) / 1e9,
                "read_gbs": calib.read_bandwidth(1 << 30) / 1e9}
    inv_w = 2.0 / measured["copy_gbs"] - 1.0 / measured["read_gbs"]
    measured["write_gbs"] = 1.0 / inv_w if inv_w > 0 else None
    log(f"measured ceilings: {measured}")
    wb = write_bytes_per_fill(dname, ch.L, M + 1)
    write_share = wb / (dbytes / args.steps) if wb is not None and dbytes > 0 else None
    for r in (roofline, roofline["other_roof"]):
        if r["bound"] != "hbm":
            r["measured_peak"] = measured["valu_int32_tops"]
        elif write_share is not None and measured["write_gbs"]:
            r["measured_peak"] = 1.0 / ((1.0 - write_share) / measured["read_gbs"]
                                        + write_share / measured["write_gbs"])
            r["write_share"] = write_share
        else:
            r["measured_peak"] = measured["copy_gbs"]
        r["frac_of_measured"] = r["achieved"] / r["measured_peak"]

    out = {
        "metric": METRIC, "value": relax / (ms_per_step * 1e-3), "unit": "relaxations/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": ch.name, "L": ch.L, "K": ch.K, "M": M, "relaxations": relax,
                   "cells": ncells, "chain_sha256": ch.sha256(), "answer": ans, "schedule_ops": nops},
        "wall_solve_ms": statistics.median(wall), "cold_solve_ms": cold_ms, "fill_ms": statistics.median(fill_ms),
        "schedule_ms": sched_ms,
        "fill_relax_per_s": relax / (statistics.median(fill_ms) * 1e-3),
        "roofline": roofline, "measured_ceilings": measured, "cpu_baseline": cpu, "tradeoff": tradeoff,
        "option_pruning": pruning, "other_workloads": others, "saving_sweep": sweep,
        "kernels": {k: {"launches_per_step": v[0] / args.steps, "ms_per_step": v[1] / args.steps,
                        "relaxations_per_step": v[2] // args.steps, "evaluated_per_step": v[3] // args.steps,
                        "table_bytes_per_step": v[4] // args.steps}
                    for k, v in kern.items()},
    }
    s.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
