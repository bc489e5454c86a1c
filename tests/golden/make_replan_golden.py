"""Write the expected re-planning decisions on full-size workloads.

Each case shifts the routing of a benchmark workload between two epochs
(`workloads.shift_routing`), takes a simple resident state as the incumbent
(`workloads.prefix_incumbent`) and runs the CPU oracle's re-planning rule.
Every stored value comes from `oracle/`; nothing here touches the HIP path.
Run from the repository root:

    python tests/golden/make_replan_golden.py [--threads T]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2608_01655_amd import workloads as W  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "replans.json")

# (case name, workload, shifted share num/den, horizon in epochs)
CASES = [("tree50k-shift50", "tree50k", 1, 2, 1000)]


def shifted(name, num, den):
    inst = W.make_workload(name)
    lam = W.shift_routing(inst.parent, inst.demand, num, den)
    inc = W.prefix_incumbent(inst.n, inst.cap)
    return inst, lam, inc


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    args = ap.parse_args()
    oracle.build(force=False)
    data = {}
    for case, name, num, den, horizon in CASES:
        inst, lam, inc = shifted(name, num, den)
        t0 = time.time()
        r = oracle.replan(inst.parent, lam, inst.recompute_cost,
                          inst.fetch_cost, inst.cap, inc, horizon,
                          n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                          order_seed=inst.order_seed, threads=args.threads)
        dt = time.time() - t0
        data[case] = {
            "workload": name, "shift": [num, den], "horizon": horizon,
            "demand_sha256": hashlib.sha256(lam.tobytes()).hexdigest(),
            "adopt": r.adopt,
            "incumbent_objective": r.incumbent_objective,
            "proposal_objective": r.proposal_objective,
            "materialization_cost": r.materialization_cost,
            "proposal_row_sha256": [hashlib.sha256(r.proposal[h].tobytes())
                                    .hexdigest() for h in range(inst.m)],
            "oracle_seconds": round(dt, 2), "oracle_threads": args.threads,
        }
        print(f"{case}: adopt {r.adopt} G {r.incumbent_objective} -> "
              f"{r.proposal_objective} cost {r.materialization_cost} "
              f"{dt:.1f}s", flush=True)
    with open(OUT, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
        fh.write("\n")


if __name__ == "__main__":
    main()
