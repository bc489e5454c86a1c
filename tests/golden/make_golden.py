"""Write the expected plans of the five benchmark workloads.

Every stored value comes from the CPU oracle (`oracle/`) run on the seeded
inputs of `paper_2608_01655_amd.workloads`; nothing here touches the HIP
path.  Run from the repository root:

    python tests/golden/make_golden.py [--threads T] [names...]
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

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "plans.json")


def summarize(inst, res, seconds, threads):
    rows = [hashlib.sha256(res.target[h].tobytes()).hexdigest()
            for h in range(inst.m)]
    return {
        "input_sha256": inst.checksum(),
        "n": inst.n, "m": inst.m, "cap": [int(c) for c in inst.cap],
        "n_starts": inst.n_starts, "max_rounds": inst.max_rounds,
        "order_seed": inst.order_seed,
        "objective": res.objective,
        "best_start": res.best_start,
        "standalone": [int(x) for x in res.standalone],
        "orders": res.orders.tolist(),
        "start_objective": [int(x) for x in res.start_objective],
        "start_sweeps": [int(x) for x in res.start_sweeps],
        "start_accepts": [int(x) for x in res.start_accepts],
        "updates": res.updates,
        "dp_cells": res.dp_cells,
        "target_row_sha256": rows,
        "target_row_count": [int(res.target[h].sum()) for h in range(inst.m)],
        "oracle_seconds": round(seconds, 2),
        "oracle_threads": threads,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    ap.add_argument("names", nargs="*", default=list(W.WORKLOADS))
    args = ap.parse_args()
    oracle.build(force=False)
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as fh:
            data = json.load(fh)
    for name in args.names:
        inst = W.make_workload(name)
        t0 = time.time()
        res = oracle.plan_instance(inst, threads=args.threads)
        dt = time.time() - t0
        data[name] = summarize(inst, res, dt, args.threads)
        print(f"{name}: objective {res.objective} best {res.best_start} "
              f"sweeps {res.start_sweeps.tolist()} {dt:.1f}s", flush=True)
        with open(OUT, "w") as fh:
            json.dump(data, fh, indent=1, sort_keys=True)
            fh.write("\n")


if __name__ == "__main__":
    main()
