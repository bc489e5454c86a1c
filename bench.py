"""Throughput of the PrefixPlace planner hot path on one MI355X.

One step = one full plan (standalone scores, WorkerGreedy, coordinate
refinement until no sweep improves, best start) of the tree50k workload
(n = 50,000 chunks, M = 16 workers, k = 4,096 each, 8 order-diverse starts,
source-dependent fetch costs) through the device-resident C-ABI entry point,
inputs already in HBM.  Prints one JSON line.  After the timed region a
re-planning leg (a 50% routing shift of the same workload, through the
host-array entry point) adds a "replan" object, and a real-valued leg (the
same workload in requests and milliseconds, as doubles) an "f64" object;
--no-replan and --no-f64 skip them.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# Algorithmic bytes per DP cell in the table formulation of Theorem 1:
# 8 B write of D[i][j], 8 B read of the skip operand D[next(i)][j], and one
# choice bit (row i+1 is produced the step before and held on chip).
BYTES_PER_CELL = 16.125
HBM_PEAK_GBS = 8000.0
METRIC = ("full PrefixPlace plans/sec and tree-DP cells/sec "
          "(n·k·updates/s), 1 GPU")
# Paper context: n = 50,000, M = 16 solved in 12.29 s on one EPYC 9V74 with
# k = 128 (Sec. V, RQ5) -- a different capacity, so not a like-for-like
# baseline.
PAPER_CONTEXT = "n=50,000, M=16, k=128: 12.29 s per plan on one EPYC 9V74"

# HBM traffic of the DP sweep as measured by hardware counters (FETCH_SIZE
# and WRITE_SIZE per dispatch, each scaled by what the same counter reads for
# a device copy of known size).  The summary records a digest of the sources
# that decide the kernel and its launch; a different digest means the
# counters describe another kernel and the figure is not reported.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_dp_hbm_traffic.md")
KERNEL_SOURCES = ("paper_2608_01655_amd/csrc/pp_kernels.hip",
                  "paper_2608_01655_amd/csrc/pp_internal.h",
                  "paper_2608_01655_amd/csrc/pp_host.cpp")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_sources_digest():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per DP-sweep launch from the committed counter summary, or
    None if there is none for this workload and these kernel sources."""
    try:
        with open(TRAFFIC_FILE) as fh:
            text = fh.read()
    except OSError:
        return None
    for m in re.finditer(r"<!-- traffic (\{.*?\}) -->", text):
        rec = json.loads(m.group(1))
        if rec.get("workload") == workload and \
                rec.get("sources_sha256") == kernel_sources_digest():
            return float(rec["bytes_per_launch"])
    return None


def copy_probe(mib):
    """A device-to-device copy of known size, for calibrating the HBM byte
    counters (run under rocprofv3 --pmc)."""
    import torch

    n = mib * 2 ** 20 // 8
    a = torch.arange(n, dtype=torch.int64, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    ok = bool(torch.equal(a, b))
    print(json.dumps({"copy_bytes": n * 8, "copies": 3, "equal": ok}),
          flush=True)
    return 0 if ok else 1


def host_description():
    """CPU model, logical CPUs and memory of the machine the bench runs on."""
    model, mem_kib = None, None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
        with open("/proc/meminfo") as fh:
            for line in fh:
                if line.startswith("MemTotal"):
                    mem_kib = int(line.split()[1])
                    break
    except OSError:
        pass
    return {"cpu_model": model, "host_cpus": os.cpu_count(),
            "mem_gib": round(mem_kib / 2 ** 20, 1) if mem_kib else None}


def cpu_baseline(inst, cells_per_plan, threads):
    """The oracle as it stands, on a bounded sample of the same workload:
    the standalone pass and the greedy pass of every start (no refinement
    sweeps), timed on the host cores."""
    import oracle

    oracle.lib()
    t0 = time.perf_counter()
    res = oracle.plan_instance(inst, flags=oracle.F_NO_REFINE, threads=threads)
    dt = time.perf_counter() - t0
    cps = res.dp_cells / dt
    return {
        "value": cps / cells_per_plan,
        "unit": "plans/s",
        "cells_per_s": cps,
        "cores": threads,
        "kind": "oracle",
        "sample": (f"{inst.name}: standalone + greedy pass of all "
                   f"{inst.n_starts} starts ({res.updates} worker updates, "
                   f"{res.dp_cells:.3e} DP cells) in {dt:.1f} s; plans/s = "
                   f"cells/s / cells of one full plan"),
        **host_description(),
    }


def replan_leg(B, W, inst, steps, warmup):
    """Epoch re-planning (Sec. IV-D) after a 50% routing shift, the incumbent
    being the first k_h preorder chunks of every worker, horizon 1,000
    epochs: the host-array entry point, so the time includes the PCIe copies
    of the inputs and outputs (inputs: demand, costs and incumbent; outputs:
    target and proposal)."""
    lam = W.shift_routing(inst.parent, inst.demand, 1, 2)
    inc = W.prefix_incumbent(inst.n, inst.cap)
    horizon = 1000

    def call():
        return B.pp_replan(inst.parent, lam, inst.recompute_cost,
                           inst.fetch_cost, inst.cap, inc, horizon,
                           n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                           order_seed=inst.order_seed)

    for _ in range(warmup):
        call()
    t0 = time.perf_counter()
    for _ in range(steps):
        r = call()
    dt = (time.perf_counter() - t0) / steps
    out = {"ms_per_replan": dt * 1e3, "includes_pcie": True,
           "shift": "50% routing shift", "horizon": horizon,
           "adopt": r.adopt, "incumbent_objective": r.incumbent_objective,
           "proposal_objective": r.proposal_objective,
           "materialization_cost": r.materialization_cost}
    gain = r.proposal_objective - r.incumbent_objective
    if gain > 0:
        out["break_even_epochs"] = r.materialization_cost // gain + 1
    gold_path = os.path.join(ROOT, "tests", "golden", "replans.json")
    if os.path.exists(gold_path):
        with open(gold_path) as fh:
            gold = json.load(fh).get(f"{inst.name}-shift50")
        if gold:
            out["parity_vs_golden"] = (
                r.adopt == gold["adopt"]
                and r.proposal_objective == gold["proposal_objective"]
                and r.incumbent_objective == gold["incumbent_objective"]
                and r.materialization_cost == gold["materialization_cost"])
    return out


def f64_leg(B, W, inst, ctx, steps, warmup):
    """The same workload in the paper's own units, as doubles (requests per
    epoch and milliseconds, each entry jittered), planned through the
    real-valued device entry point with epsilon = 1e-9 of sum(demand *
    recompute cost); inputs already in HBM."""
    import numpy as np
    import torch

    lam, w, f = W.real_valued(inst, 1)
    eps = 1e-9 * float(np.sum(lam * w))
    dev = torch.device("cuda:0")
    tl = torch.from_numpy(lam).to(dev)
    tw = torch.from_numpy(w).to(dev)
    tf = torch.from_numpy(f).to(dev)
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)

    def call(flags=0):
        return ctx.pp_plan_f64_device(inst.parent, tl, tw, tf, inst.cap, tgt,
                                      epsilon=eps, n_starts=inst.n_starts,
                                      max_rounds=inst.max_rounds,
                                      order_seed=inst.order_seed, flags=flags)

    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    plans = [call(B.PP_F_TIME_KERNELS) for _ in range(steps)]
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    p = plans[-1]
    dp_ms = sum(q.dp_kernel_ms for q in plans)
    launches = sum(q.dp_launches for q in plans)
    out = {"plans_per_s": 1.0 / dt, "ms_per_plan": dt * 1e3,
           "dp_avg_launch_ms": dp_ms / launches,
           "dp_launches_per_plan": launches // steps,
           "dp_cells_per_s_in_kernel":
               sum(q.dp_cells_executed for q in plans) / (dp_ms / 1e3),
           "objective": p.objective, "epsilon": eps,
           "sweeps_per_start": p.start_sweeps.tolist(),
           "units": "requests/epoch and ms, per-entry jitter U[0.75, 1.25]"}
    gold_path = os.path.join(ROOT, "tests", "golden", "plans_f64.json")
    if os.path.exists(gold_path):
        with open(gold_path) as fh:
            gold = json.load(fh).get(inst.name)
        if gold:
            out["parity_vs_golden"] = all(
                q.best_start == gold["best_start"]
                and q.start_sweeps.tolist() == gold["start_sweeps"]
                and abs(q.objective - float.fromhex(gold["objective"]))
                <= 1e-12 * abs(q.objective) for q in plans)
    return out


def paper_config_leg(B, W, ctx, steps, with_oracle):
    """The configuration of the paper's own timing (n = 50,000, M = 16,
    k = 128 per worker): the tree50k tree and demand with every capacity
    set to 128, in requests per epoch and milliseconds as doubles, 8
    starts, refinement to convergence, through the real-valued device entry
    point.  The paper reports 12.29 s per plan on one EPYC 9V74 for its own
    inputs of this size; the CPU oracle (one thread, the full DP table) is
    timed on the same inputs as a second point of reference."""
    import dataclasses

    import numpy as np
    import torch

    inst = W.make_workload("tree50k")
    inst = dataclasses.replace(inst, cap=np.full(inst.m, 128, np.int32))
    lam, w, f = W.real_valued(inst, 1)
    eps = 1e-9 * float(np.sum(lam * w))
    dev = torch.device("cuda:0")
    tl = torch.from_numpy(lam).to(dev)
    tw = torch.from_numpy(w).to(dev)
    tf = torch.from_numpy(f).to(dev)
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)
    kw = dict(epsilon=eps, n_starts=inst.n_starts, max_rounds=inst.max_rounds,
              order_seed=inst.order_seed)
    ctx.pp_plan_f64_device(inst.parent, tl, tw, tf, inst.cap, tgt, **kw)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        p = ctx.pp_plan_f64_device(inst.parent, tl, tw, tf, inst.cap, tgt, **kw)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    out = {"workload": "tree50k tree and demand, k = 128 for all 16 workers, "
                       "real-valued (requests, ms)",
           "ms_per_plan": dt * 1e3, "updates_per_plan": p.updates,
           "sweeps_per_start": p.start_sweeps.tolist(), "objective": p.objective,
           "paper_s_per_plan": 12.29, "paper_hardware": "one EPYC 9V74",
           "ratio_paper_time_to_this": 12.29 / dt}
    if with_oracle:
        import oracle

        oracle.lib()
        t1 = time.perf_counter()
        o = oracle.plan_f64(inst.parent, lam, w, f, inst.cap, **kw)
        out["oracle_s_per_plan_1_thread"] = time.perf_counter() - t1
        out["same_as_oracle"] = (
            bool(np.array_equal(o.target, tgt.cpu().numpy()))
            and abs(o.objective - p.objective) <= 1e-12 * abs(o.objective))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="tree50k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--safeguards", action="store_true",
                    help="requester-side variant of the workload (each "
                         "requester's fetch cost taken from one source) "
                         "planned with the comparator safeguards")
    ap.add_argument("--no-replan", action="store_true",
                    help="skip the re-planning leg")
    ap.add_argument("--no-host-plan", action="store_true",
                    help="skip the timing of the host-array entry point")
    ap.add_argument("--no-f64", action="store_true",
                    help="skip the real-valued leg")
    ap.add_argument("--no-paper-config", action="store_true",
                    help="skip the leg at the paper's own timing configuration")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device (counter "
                         "calibration) and exit")
    args = ap.parse_args()
    if args.copy_probe:
        sys.exit(copy_probe(args.copy_probe))
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the planner's starts would "
              "shard across GPUs with one exchange of (objective, start) "
              "pairs, which this build does not run", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_01655_amd import binding as B
    from paper_2608_01655_amd import workloads as W

    if not os.path.exists(B.LIB_PATH):
        from paper_2608_01655_amd import build

        build.build()
    inst = W.make_workload(args.workload)
    plan_flags = 0
    if args.safeguards:
        import dataclasses

        f_req = inst.fetch_cost.copy()
        for dst in range(inst.m):
            src0 = 1 if dst == 0 else 0
            for src in range(inst.m):
                if src != dst and inst.m > 1:
                    f_req[src, dst] = inst.fetch_cost[src0, dst]
        inst = dataclasses.replace(inst, name=inst.name + "-requester-side",
                                   fetch_cost=f_req)
        plan_flags = B.PP_F_SAFEGUARDS
    log(f"[bench] workload {inst.name}: n={inst.n} m={inst.m} "
        f"k={int(inst.cap.min())}..{int(inst.cap.max())} S={inst.n_starts}")
    dev = torch.device("cuda:0")
    lam = torch.from_numpy(inst.demand).to(dev)
    w = torch.from_numpy(inst.recompute_cost).to(dev)
    f = torch.from_numpy(inst.fetch_cost).to(dev)
    tgt = torch.zeros((inst.m, inst.n), dtype=torch.uint8, device=dev)
    ctx = B.Context(0)

    def step(flags=0):
        return ctx.pp_plan_device(inst.parent, lam, w, f, inst.cap, tgt,
                                  n_starts=inst.n_starts,
                                  max_rounds=inst.max_rounds,
                                  order_seed=inst.order_seed,
                                  flags=flags | plan_flags)

    for i in range(args.warmup):
        p = step()
        log(f"[bench] warmup {i}: objective {p.objective}")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    plans, marks = [], []
    for i in range(args.steps):
        plans.append(step(B.PP_F_TIME_KERNELS))
        marks.append(time.perf_counter())  # the call returns after its stream drained
        log(f"[bench] step {i}: objective {plans[-1].objective} "
            f"dp {plans[-1].dp_kernel_ms:.1f} ms")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    step_ms = sorted((b - a) * 1e3 for a, b in zip([t0] + marks[:-1], marks))
    p = plans[-1]
    objectives = {q.objective for q in plans}
    gold_ok = None
    gold_path = os.path.join(ROOT, "tests", "golden", "plans.json")
    if os.path.exists(gold_path):
        with open(gold_path) as fh:
            gold = json.load(fh).get(inst.name)
        if gold:
            gold_ok = objectives == {gold["objective"]}
    cells = p.dp_cells
    plans_per_s = args.steps / dt
    cells_per_s = cells * args.steps / dt
    # cells the sweeps actually processed (refinement updates of workers
    # whose inputs did not change are resolved without a sweep)
    exec_cells = sum(q.dp_cells_executed for q in plans)
    dp_ms = sum(q.dp_kernel_ms for q in plans)
    launches = sum(q.dp_launches for q in plans)
    bytes_per_launch = exec_cells * BYTES_PER_CELL / launches
    avg_launch_s = dp_ms / launches / 1e3
    achieved = bytes_per_launch / avg_launch_s / 1e9
    traffic = measured_traffic(inst.name)
    out = {
        "metric": METRIC,
        "value": plans_per_s,
        "unit": "plans/s",
        "dp_cells_per_s": cells_per_s,
        "dp_cells_executed_per_s": exec_cells / dt,
        # model fraction on the cells actually swept
        "dp_cells_per_s_frac_hbm_roofline":
            exec_cells / dt * BYTES_PER_CELL / (HBM_PEAK_GBS * 1e9),
        "plans_per_s_frac_hbm_roofline":
            exec_cells / dt * BYTES_PER_CELL / (HBM_PEAK_GBS * 1e9),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt / args.steps * 1e3,
        "ms_per_step_median": step_ms[len(step_ms) // 2],
        "ms_per_step_min": step_ms[0],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": inst.name, "n": inst.n, "workers": inst.m,
            "k": [int(x) for x in sorted(set(inst.cap.tolist()))],
            "starts": inst.n_starts, "max_rounds": inst.max_rounds,
            "updates_per_plan": p.updates, "dp_cells_per_plan": cells,
            "dp_cells_executed_per_plan": exec_cells // args.steps,
            "sweeps_per_start": p.start_sweeps.tolist(),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "k_dp (rooted-tree DP sweep)",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            # the same launches against the bytes the counters saw move
            "measured_frac": (traffic / avg_launch_s / 1e9 / HBM_PEAK_GBS
                              if traffic else None),
            "bytes_per_cell": BYTES_PER_CELL,
            "dp_launches_per_plan": launches // args.steps,
            "avg_launch_ms": avg_launch_s * 1e3,
            "dp_cells_per_s_in_kernel": exec_cells / (dp_ms / 1e3),
            "dp_share_of_plan_time": dp_ms / 1e3 / dt,
        },
        "parity_vs_golden": gold_ok,
        **({"safeguards": {"run": p.safeguards_run, "returned": p.best_start,
                           "objectives": list(p.safeguard_objective)}}
           if args.safeguards else {}),
        "paper_context": PAPER_CONTEXT,
    }
    # the host-array entry point on the same inputs: PCIe copies of the
    # inputs and the placement inside the call
    host_ms = []
    for _ in range(0 if args.no_host_plan else 2):
        t1 = time.perf_counter()
        hp = B.pp_plan(inst.parent, inst.demand, inst.recompute_cost,
                       inst.fetch_cost, inst.cap, n_starts=inst.n_starts,
                       max_rounds=inst.max_rounds, order_seed=inst.order_seed,
                       flags=plan_flags)
        host_ms.append((time.perf_counter() - t1) * 1e3)
    if host_ms:
        out["host_pp_plan_ms"] = min(host_ms)
        out["host_pp_plan_same_objective"] = hp.objective == p.objective
    if not args.no_replan and not args.safeguards:
        log("[bench] re-planning leg")
        out["replan"] = replan_leg(B, W, inst, max(1, min(args.steps, 3)),
                                   min(args.warmup, 1))
    if not args.no_f64 and not args.safeguards:
        log("[bench] real-valued leg")
        out["f64"] = f64_leg(B, W, inst, ctx, max(1, min(args.steps, 3)),
                             min(args.warmup, 1))
    if not args.no_paper_config and not args.safeguards:
        log("[bench] paper-configuration leg (k = 128)")
        out["paper_config"] = paper_config_leg(B, W, ctx, max(1, min(args.steps, 3)),
                                                not args.no_cpu_baseline)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        threads = max(1, min(8, os.cpu_count() or 1))
        out["cpu_baseline"] = cpu_baseline(inst, cells, threads)
    ctx.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
