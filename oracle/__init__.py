"""ctypes wrapper of the plain CPU oracle (pporacle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the package smoke check
and by the bench's CPU-baseline leg.  The product path never imports it.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "pporacle.c")
LIB = os.path.join(_HERE, "libpporacle.so")

OK, E_ARG, E_TREE, E_RANGE, E_OVERFLOW, E_NOMEM = 0, -1, -2, -3, -4, -5
F_NO_REFINE = 2
F_SAFEGUARDS = 8


def build(force: bool = True) -> str:
    """Compile the oracle with the host C compiler (no GPU code)."""
    if force or not os.path.exists(LIB) or \
            os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        # no contraction of a*b + c into one rounding: the real-valued
        # entry points round every product and sum as written
        subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra",
                        "-ffp-contract=off", "-shared", "-fPIC", "-pthread",
                        "-o", tmp, SRC],
                       check=True)
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=False)
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32, i64, u32, u64 = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                              ctypes.c_uint64)
        L.ppo_preorder.argtypes = [i32, P, P, P]
        L.ppo_rooted_dp.argtypes = [i32, P, P, i32, P, P]
        L.ppo_marginal.argtypes = [i32, i32, P, P, P, P, i32, P, P]
        L.ppo_objective.argtypes = [i32, i32, P, P, P, P, P]
        L.ppo_orders.argtypes = [i32, i32, u64, P, P]
        L.ppo_num_starts.argtypes = [i32, i32]
        L.ppo_num_starts.restype = i32
        L.ppo_splitmix64_stream.argtypes = [u64, i32, P]
        L.ppo_splitmix64_stream.restype = None
        L.ppo_plan.argtypes = [i32, i32, P, P, P, P, P, i32, i32, u64, P, u32,
                               i32, P, P, P, P, P, P, P, P, P]
        L.ppo_requester_side.argtypes = [i32, i32, P]
        f64 = ctypes.c_double
        L.ppo_rooted_dp_f64.argtypes = [i32, P, P, i32, P, P]
        L.ppo_marginal_f64.argtypes = [i32, i32, P, P, P, P, i32, P]
        L.ppo_objective_f64.argtypes = [i32, i32, P, P, P, P, P]
        L.ppo_plan_f64.argtypes = [i32, i32, P, P, P, P, P, f64, i32, i32, u64,
                                   P, u32, P, P, P, P, P, P, P, P, P]
        L.ppo_replan_f64.argtypes = [i32, i32, P, P, P, P, P, P, f64, f64, i32,
                                     i32, u64, u32, P, P, P, P]
        L.ppo_candidates.argtypes = [i32, i32, P, P, P, P, P, P, P]
        L.ppo_materialization_cost.argtypes = [i32, i32, P, P, P, P, P]
        L.ppo_replan.argtypes = [i32, i32, P, P, P, P, P, P, i64, i32, i32,
                                 u64, u32, i32, P, P, P]
        for f in (L.ppo_preorder, L.ppo_rooted_dp, L.ppo_marginal,
                  L.ppo_objective, L.ppo_orders, L.ppo_plan,
                  L.ppo_requester_side, L.ppo_candidates,
                  L.ppo_materialization_cost, L.ppo_replan):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle returned {code}")
        self.code = code


def _check(rc: int):
    if rc != OK:
        raise OracleError(rc)


def preorder(parent):
    parent = _c(parent, np.int32)
    n = parent.shape[0]
    order = np.empty(n, np.int32)
    nxt = np.empty(n, np.int32)
    _check(lib().ppo_preorder(n, _p(parent), _p(order), _p(nxt)))
    return order, nxt


def rooted_dp(parent, profit, k):
    parent = _c(parent, np.int32)
    profit = _c(profit, np.int64)
    n = parent.shape[0]
    sel = np.zeros(n, np.uint8)
    val = np.zeros(1, np.int64)
    _check(lib().ppo_rooted_dp(n, _p(parent), _p(profit), int(k), _p(sel),
                               _p(val)))
    return sel, int(val[0])


def marginal(demand, recompute_cost, fetch_cost, target, h):
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    target = _c(target, np.uint8)
    m, n = demand.shape
    prof = np.zeros(n, np.int64)
    g = np.zeros(1, np.int64)
    _check(lib().ppo_marginal(n, m, _p(demand), _p(w), _p(f), _p(target),
                              int(h), _p(prof), _p(g)))
    return prof, int(g[0])


def objective(demand, recompute_cost, fetch_cost, target) -> int:
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    target = _c(target, np.uint8)
    m, n = demand.shape
    out = np.zeros(1, np.int64)
    _check(lib().ppo_objective(n, m, _p(demand), _p(w), _p(f), _p(target),
                               _p(out)))
    return int(out[0])


def requester_side(fetch_cost) -> bool:
    """Reading R18: fetch_cost[src][dst][b] equal over every src != dst."""
    f = _c(fetch_cost, np.int64)
    m, n = f.shape[0], f.shape[2]
    return bool(lib().ppo_requester_side(n, m, _p(f)))


def candidates(parent, demand, recompute_cost, fetch_cost, cap):
    """The Independent, Popularity and LocalDedup placements (reading R15)
    as uint8 [3][m][n] and their objectives."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    cap = _c(cap, np.int32)
    m, n = demand.shape
    tg = np.zeros((3, m, n), np.uint8)
    objs = np.zeros(3, np.int64)
    _check(lib().ppo_candidates(n, m, _p(parent), _p(demand), _p(w), _p(f),
                                _p(cap), _p(tg), _p(objs)))
    return tg, [int(x) for x in objs]


def num_starts(m: int, n_starts: int) -> int:
    return int(lib().ppo_num_starts(m, n_starts))


def orders(m, n_starts, order_seed, standalone):
    st = _c(standalone, np.int64)
    S = num_starts(m, n_starts)
    out = np.zeros((S, m), np.int32)
    _check(lib().ppo_orders(m, n_starts, ctypes.c_uint64(order_seed & (2**64 - 1)),
                            _p(st), _p(out)))
    return out


def splitmix64_stream(seed: int, count: int) -> list[int]:
    out = np.zeros(count, np.uint64)
    lib().ppo_splitmix64_stream(ctypes.c_uint64(seed), count, _p(out))
    return [int(x) for x in out]


@dataclass
class PlanResult:
    target: np.ndarray          # uint8 [m][n]
    objective: int
    standalone: np.ndarray      # int64 [m]
    orders: np.ndarray          # int32 [S][m]
    start_objective: np.ndarray
    start_sweeps: np.ndarray
    start_accepts: np.ndarray
    best_start: int             # start index, or S + c for safeguard c
    updates: int
    dp_cells: int
    safeguards_run: bool = False
    safeguard_objective: tuple = (0, 0, 0)


def plan(parent, demand, recompute_cost, fetch_cost, cap, *, n_starts=1,
         max_rounds=0, order_seed=0, orders_in=None, flags=0, threads=1
         ) -> PlanResult:
    parent = _c(parent, np.int32)
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    cap = _c(cap, np.int32)
    m, n = demand.shape
    S = num_starts(m, n_starts)
    if orders_in is not None:
        orders_in = _c(orders_in, np.int32)
    tgt = np.zeros((m, n), np.uint8)
    obj = np.zeros(1, np.int64)
    st = np.zeros(m, np.int64)
    ords = np.zeros((S, m), np.int32)
    so = np.zeros(S, np.int64)
    ss = np.zeros(S, np.int32)
    sa = np.zeros(S, np.int32)
    info = np.zeros(5, np.int64)
    sgo = np.zeros(3, np.int64)
    _check(lib().ppo_plan(n, m, _p(parent), _p(demand), _p(w), _p(f), _p(cap),
                          int(n_starts), int(max_rounds),
                          ctypes.c_uint64(order_seed & (2**64 - 1)),
                          _p(orders_in), int(flags), int(threads), _p(tgt),
                          _p(obj), _p(st), _p(ords), _p(so), _p(ss), _p(sa),
                          _p(info), _p(sgo)))
    return PlanResult(target=tgt, objective=int(obj[0]), standalone=st,
                      orders=ords, start_objective=so, start_sweeps=ss,
                      start_accepts=sa, best_start=int(info[0]),
                      updates=int(info[1]), dp_cells=int(info[2]),
                      safeguards_run=bool(info[4]),
                      safeguard_objective=tuple(int(x) for x in sgo))


def materialization_cost(recompute_cost, fetch_cost, incumbent, proposal) -> int:
    """Reading R21: one-time cost of the proposal's chunks that the
    incumbent does not hold at the same worker."""
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    inc = _c(incumbent, np.uint8)
    prop = _c(proposal, np.uint8)
    m, n = w.shape
    out = np.zeros(1, np.int64)
    _check(lib().ppo_materialization_cost(n, m, _p(w), _p(f), _p(inc), _p(prop),
                                          _p(out)))
    return int(out[0])


@dataclass
class ReplanResult:
    target: np.ndarray          # the placement to use
    proposal: np.ndarray        # the re-optimized plan
    adopt: bool
    incumbent_objective: int
    proposal_objective: int
    materialization_cost: int


def replan(parent, demand, recompute_cost, fetch_cost, cap, incumbent, horizon,
           *, n_starts=1, max_rounds=0, order_seed=0, flags=0, threads=1
           ) -> ReplanResult:
    """Epoch re-planning (Sec. IV-D; readings R21, R22)."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    cap = _c(cap, np.int32)
    inc = _c(incumbent, np.uint8)
    m, n = demand.shape
    tgt = np.zeros((m, n), np.uint8)
    prop = np.zeros((m, n), np.uint8)
    res = np.zeros(4, np.int64)
    _check(lib().ppo_replan(n, m, _p(parent), _p(demand), _p(w), _p(f), _p(cap),
                            _p(inc), int(horizon), int(n_starts), int(max_rounds),
                            ctypes.c_uint64(order_seed & (2**64 - 1)), int(flags),
                            int(threads), _p(tgt), _p(prop), _p(res)))
    return ReplanResult(target=tgt, proposal=prop, adopt=bool(res[0]),
                        incumbent_objective=int(res[1]),
                        proposal_objective=int(res[2]),
                        materialization_cost=int(res[3]))


def plan_instance(inst, **kw) -> PlanResult:
    """Plan a `workloads.Instance` with its own start/round/seed settings."""
    args = dict(n_starts=inst.n_starts, max_rounds=inst.max_rounds,
                order_seed=inst.order_seed)
    args.update(kw)
    return plan(inst.parent, inst.demand, inst.recompute_cost, inst.fetch_cost,
                inst.cap, **args)


# ------------------------------------------------------ real-valued costs

def rooted_dp_f64(parent, profit, k):
    """Eq. 9 on doubles (reading R24)."""
    parent = _c(parent, np.int32)
    profit = _c(profit, np.float64)
    n = parent.shape[0]
    sel = np.zeros(n, np.uint8)
    val = np.zeros(1, np.float64)
    _check(lib().ppo_rooted_dp_f64(n, _p(parent), _p(profit), int(k), _p(sel),
                                   _p(val)))
    return sel, float(val[0])


def marginal_f64(demand, recompute_cost, fetch_cost, target, h):
    """Eq. 7 on doubles, requester terms summed in increasing m."""
    demand = _c(demand, np.float64)
    w = _c(recompute_cost, np.float64)
    f = _c(fetch_cost, np.float64)
    target = _c(target, np.uint8)
    m, n = demand.shape
    prof = np.zeros(n, np.float64)
    _check(lib().ppo_marginal_f64(n, m, _p(demand), _p(w), _p(f), _p(target),
                                  int(h), _p(prof)))
    return prof


def objective_f64(demand, recompute_cost, fetch_cost, target) -> float:
    """Eq. 6 on doubles, b outer, m inner."""
    demand = _c(demand, np.float64)
    w = _c(recompute_cost, np.float64)
    f = _c(fetch_cost, np.float64)
    target = _c(target, np.uint8)
    m, n = demand.shape
    out = np.zeros(1, np.float64)
    _check(lib().ppo_objective_f64(n, m, _p(demand), _p(w), _p(f), _p(target),
                                   _p(out)))
    return float(out[0])


@dataclass
class PlanF64Result:
    target: np.ndarray          # uint8 [m][n]
    objective: float
    standalone: np.ndarray      # float64 [m]
    orders: np.ndarray          # int32 [S][m]
    start_objective: np.ndarray  # float64 [S]
    start_sweeps: np.ndarray
    start_accepts: np.ndarray
    best_start: int
    updates: int
    dp_cells: int
    safeguards_run: bool = False
    safeguard_objective: tuple = (0.0, 0.0, 0.0)


def plan_f64(parent, demand, recompute_cost, fetch_cost, cap, *, epsilon=0.0,
             n_starts=1, max_rounds=0, order_seed=0, orders_in=None, flags=0
             ) -> PlanF64Result:
    """Algorithm 1 on real-valued costs with refinement tolerance epsilon
    (reading R24)."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.float64)
    w = _c(recompute_cost, np.float64)
    f = _c(fetch_cost, np.float64)
    cap = _c(cap, np.int32)
    m, n = demand.shape
    S = num_starts(m, n_starts)
    if orders_in is not None:
        orders_in = _c(orders_in, np.int32)
    tgt = np.zeros((m, n), np.uint8)
    obj = np.zeros(1, np.float64)
    st = np.zeros(m, np.float64)
    ords = np.zeros((S, m), np.int32)
    so = np.zeros(S, np.float64)
    ss = np.zeros(S, np.int32)
    sa = np.zeros(S, np.int32)
    info = np.zeros(5, np.int64)
    sgo = np.zeros(3, np.float64)
    _check(lib().ppo_plan_f64(n, m, _p(parent), _p(demand), _p(w), _p(f),
                              _p(cap), float(epsilon), int(n_starts),
                              int(max_rounds),
                              ctypes.c_uint64(order_seed & (2**64 - 1)),
                              _p(orders_in), int(flags), _p(tgt), _p(obj),
                              _p(st), _p(ords), _p(so), _p(ss), _p(sa),
                              _p(info), _p(sgo)))
    return PlanF64Result(target=tgt, objective=float(obj[0]), standalone=st,
                         orders=ords, start_objective=so, start_sweeps=ss,
                         start_accepts=sa, best_start=int(info[0]),
                         updates=int(info[1]), dp_cells=int(info[2]),
                         safeguards_run=bool(info[4]),
                         safeguard_objective=tuple(float(x) for x in sgo))


@dataclass
class ReplanF64Result:
    target: np.ndarray
    proposal: np.ndarray
    adopt: bool
    incumbent_objective: float
    proposal_objective: float
    materialization_cost: float


def replan_f64(parent, demand, recompute_cost, fetch_cost, cap, incumbent,
               horizon, *, epsilon=0.0, n_starts=1, max_rounds=0, order_seed=0,
               flags=0) -> ReplanF64Result:
    """Epoch re-planning on real-valued costs (readings R21, R22, R24)."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.float64)
    w = _c(recompute_cost, np.float64)
    f = _c(fetch_cost, np.float64)
    cap = _c(cap, np.int32)
    inc = _c(incumbent, np.uint8)
    m, n = demand.shape
    tgt = np.zeros((m, n), np.uint8)
    prop = np.zeros((m, n), np.uint8)
    adopt = np.zeros(1, np.int32)
    res = np.zeros(3, np.float64)
    _check(lib().ppo_replan_f64(n, m, _p(parent), _p(demand), _p(w), _p(f),
                                _p(cap), _p(inc), float(horizon), float(epsilon),
                                int(n_starts), int(max_rounds),
                                ctypes.c_uint64(order_seed & (2**64 - 1)),
                                int(flags), _p(tgt), _p(prop), _p(adopt), _p(res)))
    return ReplanF64Result(target=tgt, proposal=prop, adopt=bool(adopt[0]),
                           incumbent_objective=float(res[0]),
                           proposal_objective=float(res[1]),
                           materialization_cost=float(res[2]))
