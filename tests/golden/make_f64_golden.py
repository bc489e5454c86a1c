"""Write the expected real-valued plan of the 50,000-chunk benchmark tree.

The workload's inputs in the paper's own units (`workloads.real_valued`,
seed 1: requests per epoch and milliseconds, each entry jittered), planned
by the CPU oracle's real-valued planner with the benchmark's start settings
and epsilon = 1e-9 of the sum of demand times recompute cost.  Nothing here
touches the HIP path.  Run from the repository root (single-threaded, about
half an hour):

    python tests/golden/make_f64_golden.py
"""

from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2608_01655_amd import workloads as W  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "plans_f64.json")


def case(name):
    inst = W.make_workload(name)
    lam, w, f = W.real_valued(inst, 1)
    eps = 1e-9 * float(np.sum(lam * w))
    return inst, lam, w, f, eps


def main():
    oracle.build(force=False)
    data = {}
    for name in ("tree50k",):
        inst, lam, w, f, eps = case(name)
        t0 = time.time()
        r = oracle.plan_f64(inst.parent, lam, w, f, inst.cap, epsilon=eps,
                            n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                            order_seed=inst.order_seed)
        dt = time.time() - t0
        data[name] = {
            "inputs_sha256": hashlib.sha256(lam.tobytes() + w.tobytes() +
                                            f.tobytes()).hexdigest(),
            "epsilon": eps.hex(),
            "objective": r.objective.hex(),
            "best_start": r.best_start,
            "standalone": [x.hex() for x in r.standalone.tolist()],
            "orders": r.orders.tolist(),
            "start_objective": [x.hex() for x in r.start_objective.tolist()],
            "start_sweeps": r.start_sweeps.tolist(),
            "start_accepts": r.start_accepts.tolist(),
            "updates": r.updates, "dp_cells": r.dp_cells,
            "target_row_sha256": [hashlib.sha256(r.target[h].tobytes()).hexdigest()
                                  for h in range(inst.m)],
            "oracle_seconds": round(dt, 1),
        }
        print(f"{name}: objective {r.objective} best {r.best_start} sweeps "
              f"{r.start_sweeps.tolist()} {dt:.0f}s", flush=True)
    with open(OUT, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
        fh.write("\n")


if __name__ == "__main__":
    main()
