"""Write the oracle's results for a full-size benchmark chain: per-row digests of its
Opt and choice tables, its answer and its schedule (tests/golden/config<N>_*.*).

Only the CPU oracle (oracle/) computes anything stored here; the chain comes from the
seeded generator.  Usage: python tests/golden/make_config_digests.py 4
(configuration 4: L=384, K=16, M=6000 takes about 8 minutes and 6 GB of memory on one
core).
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

import oracle  # noqa: E402
from paper_2307_01236_amd.chaingen import make_config_chain  # noqa: E402
from rowdigest import arg_digests, opt_digests  # noqa: E402


def main(cfg: int) -> None:
    ch = make_config_chain(cfg)
    t0 = time.perf_counter()
    sol = oracle.solve(ch)
    secs = time.perf_counter() - t0
    print(f"{ch.name}: oracle {secs:.1f} s, answer {sol.answer}", flush=True)
    answer = sol.answer
    sched = oracle.schedule(sol) if answer != oracle.INF else None
    opt, arg = sol.rows()
    del sol
    od = opt_digests(opt)
    ad = arg_digests(arg)
    np.savez(os.path.join(HERE, f"config{cfg}_row_digests.npz"), opt=od, arg=ad)
    meta = {
        "config": cfg,
        "workload": ch.name,
        "L": ch.L, "K": ch.K, "M": ch.M,
        "chain_sha256": ch.sha256(),
        "answer": answer,
        "oracle_seconds_one_core": round(secs, 1),
        "n_fwd": None if sched is None else sched[1],
        "schedule": None if sched is None else sched[0].tolist(),
        "digest": "per-row CRC-32, tests/rowdigest.py",
        "written_by": "tests/golden/make_config_digests.py (CPU oracle only)",
    }
    with open(os.path.join(HERE, f"config{cfg}_oracle.json"), "w") as f:
        json.dump(meta, f)
        f.write("\n")


if __name__ == "__main__":
    main(int(sys.argv[1]) if len(sys.argv) > 1 else 4)
