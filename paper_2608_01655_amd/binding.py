"""Thin ctypes binding of libprefixplace.so (include/prefixplace.h).

Argument marshalling only: every step of the planner runs in the library's
gfx950 kernels.  Names follow the C ABI.  The binding refuses to run if the
built library is missing -- there is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libprefixplace.so")

PP_OK, PP_E_ARG, PP_E_TREE, PP_E_RANGE, PP_E_OVERFLOW = 0, -1, -2, -3, -4
PP_E_NOMEM, PP_E_DEVICE, PP_E_UNSUPPORTED = -5, -6, -7
PP_F_VALIDATE_ONLY, PP_F_NO_REFINE, PP_F_TIME_KERNELS, PP_F_SAFEGUARDS = 1, 2, 4, 8

_P = ctypes.c_void_p


class pp_options(ctypes.Structure):
    _fields_ = [("n_starts", ctypes.c_int32), ("max_rounds", ctypes.c_int32),
                ("order_seed", ctypes.c_uint64), ("orders", _P),
                ("flags", ctypes.c_uint32)]


class pp_stats(ctypes.Structure):
    _fields_ = [("best_start", ctypes.c_int32), ("n_starts", ctypes.c_int32),
                ("updates", ctypes.c_int64), ("dp_cells", ctypes.c_int64),
                ("start_objective", _P), ("start_sweeps", _P),
                ("start_accepts", _P), ("standalone", _P), ("orders", _P),
                ("dp_kernel_ms", ctypes.c_double),
                ("dp_launches", ctypes.c_int32),
                ("safeguards_run", ctypes.c_int32),
                ("safeguard_objective", ctypes.c_int64 * 3),
                ("dp_cells_executed", ctypes.c_int64),
                ("dp_lane_cells", ctypes.c_int32),
                ("dp_fmax", ctypes.c_int32),
                ("dp_restarts", ctypes.c_int32)]


class pp_stats_f64(ctypes.Structure):
    _fields_ = [("best_start", ctypes.c_int32), ("n_starts", ctypes.c_int32),
                ("updates", ctypes.c_int64), ("dp_cells", ctypes.c_int64),
                ("start_objective", _P), ("start_sweeps", _P),
                ("start_accepts", _P), ("standalone", _P), ("orders", _P),
                ("dp_kernel_ms", ctypes.c_double),
                ("dp_launches", ctypes.c_int32),
                ("safeguards_run", ctypes.c_int32),
                ("safeguard_objective", ctypes.c_double * 3),
                ("dp_cells_executed", ctypes.c_int64),
                ("dp_lane_cells", ctypes.c_int32),
                ("dp_fmax", ctypes.c_int32),
                ("dp_restarts", ctypes.c_int32)]


class pp_replan_info(ctypes.Structure):
    _fields_ = [("adopt", ctypes.c_int32), ("incumbent_objective", ctypes.c_int64),
                ("proposal_objective", ctypes.c_int64),
                ("materialization_cost", ctypes.c_int64)]


class pp_replan_info_f64(ctypes.Structure):
    _fields_ = [("adopt", ctypes.c_int32), ("incumbent_objective", ctypes.c_double),
                ("proposal_objective", ctypes.c_double),
                ("materialization_cost", ctypes.c_double)]


class PPError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"prefixplace error {code}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load the in-tree library; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2608_01655_amd.build`")
        # PyTorch-ROCm ships its own HIP runtime (same SONAME as the system
        # one, but its libraries ask for it under another file name).  Load
        # torch first so this library binds to that same runtime instead of
        # bringing a second HIP/HSA runtime into the process.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
        L.pp_abi_version.restype = ctypes.c_int
        L.pp_last_error.restype = ctypes.c_char_p
        L.pp_num_starts.argtypes = [i32, i32]
        L.pp_num_starts.restype = i32
        L.pp_plan.argtypes = [i32, i32, _P, _P, _P, _P, _P, _P, _P, _P, _P]
        L.pp_replan.argtypes = [i32, i32, _P, _P, _P, _P, _P, _P, i64, _P, _P,
                                _P, _P, _P]
        f64 = ctypes.c_double
        L.pp_plan_f64.argtypes = [i32, i32, _P, _P, _P, _P, _P, f64, _P, _P, _P, _P]
        L.pp_plan_f64_device.argtypes = [_P, i32, i32, _P, _P, _P, _P, _P, f64, _P,
                                         _P, _P, _P, _P]
        L.pp_rooted_dp_f64.argtypes = [i32, _P, _P, i32, _P, _P]
        L.pp_replan_f64.argtypes = [i32, i32, _P, _P, _P, _P, _P, _P, f64, f64,
                                    _P, _P, _P, _P, _P]
        L.pp_rooted_dp.argtypes = [i32, _P, _P, i32, _P, _P]
        L.pp_marginal.argtypes = [i32, i32, _P, _P, _P, _P, i32, _P, _P]
        L.pp_objective.argtypes = [i32, i32, _P, _P, _P, _P, _P]
        L.pp_orders.argtypes = [i32, i32, u64, _P, _P]
        L.pp_sweep_layout.argtypes = [i32, _P, i32, _P, _P, _P]
        L.pp_sweep_layout.restype = ctypes.c_int
        L.pp_sweep_spills.argtypes = [i32, _P, _P, _P, _P, _P, _P, _P, _P, _P]
        L.pp_sweep_spills.restype = ctypes.c_int
        L.pp_backtrack_table.argtypes = [i32, _P, _P, _P]
        L.pp_backtrack_table.restype = ctypes.c_int
        L.pp_ctx_create.argtypes = [ctypes.POINTER(_P), ctypes.c_int]
        L.pp_ctx_destroy.argtypes = [_P]
        L.pp_ctx_destroy.restype = None
        L.pp_plan_device.argtypes = [_P, i32, i32, _P, _P, _P, _P, _P, _P, _P,
                                     _P, _P, _P]
        L.pp_objective_device_noalloc.argtypes = [i32, i32, _P, _P, _P, _P, _P, _P]
        for f in (L.pp_plan, L.pp_replan, L.pp_replan_f64, L.pp_plan_f64,
                  L.pp_plan_f64_device,
                  L.pp_rooted_dp_f64, L.pp_rooted_dp, L.pp_marginal, L.pp_objective,
                  L.pp_orders, L.pp_ctx_create, L.pp_plan_device,
                  L.pp_objective_device_noalloc):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def pp_abi_version() -> int:
    return int(lib().pp_abi_version())


def pp_last_error() -> str:
    return lib().pp_last_error().decode()


def _check(rc: int):
    if rc != PP_OK:
        raise PPError(rc, pp_last_error())


def _p(a):
    return None if a is None else a.ctypes.data_as(_P)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def pp_num_starts(m: int, n_starts: int) -> int:
    return int(lib().pp_num_starts(m, n_starts))


@dataclass
class Plan:
    target: object              # uint8 [m][n] (numpy, or a device tensor)
    objective: int
    best_start: int
    n_starts: int
    updates: int
    dp_cells: int
    start_objective: np.ndarray
    start_sweeps: np.ndarray
    start_accepts: np.ndarray
    standalone: np.ndarray
    orders: np.ndarray
    dp_kernel_ms: float
    dp_launches: int
    safeguards_run: bool = False
    safeguard_objective: tuple = (0, 0, 0)
    dp_cells_executed: int = 0
    dp_lane_cells: int = 0      # DP cells per lane of the sweep (1, 2, 4)
    dp_fmax: bool = False       # maximum by one 64-bit float instruction
    dp_restarts: int = 0        # plan runs repeated after a stalled sweep


def _options(m, n_starts, max_rounds, order_seed, orders, flags):
    o = pp_options()
    o.n_starts = int(n_starts)
    o.max_rounds = int(max_rounds)
    o.order_seed = int(order_seed) & (2 ** 64 - 1)
    keep = None
    if orders is not None:
        keep = _c(orders, np.int32)
        o.orders = keep.ctypes.data
    o.flags = int(flags)
    S = pp_num_starts(m, n_starts)
    st = pp_stats()
    arrs = dict(start_objective=np.zeros(S, np.int64),
                start_sweeps=np.zeros(S, np.int32),
                start_accepts=np.zeros(S, np.int32),
                standalone=np.zeros(m, np.int64),
                orders=np.zeros((S, m), np.int32))
    for k, v in arrs.items():
        setattr(st, k, v.ctypes.data)
    return o, st, arrs, keep


def _plan_from(st, arrs, target, objective):
    return Plan(target=target, objective=int(objective), best_start=st.best_start,
                n_starts=st.n_starts, updates=st.updates, dp_cells=st.dp_cells,
                dp_kernel_ms=st.dp_kernel_ms, dp_launches=st.dp_launches,
                safeguards_run=bool(st.safeguards_run),
                safeguard_objective=tuple(int(x) for x in st.safeguard_objective),
                dp_cells_executed=st.dp_cells_executed,
                dp_lane_cells=st.dp_lane_cells, dp_fmax=bool(st.dp_fmax),
                dp_restarts=st.dp_restarts, **arrs)


def pp_plan(parent, demand, recompute_cost, fetch_cost, cap, *, n_starts=8,
            max_rounds=0, order_seed=0, orders=None, flags=0) -> Plan:
    """Host-array planner call (see pp_plan in include/prefixplace.h)."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    cap = _c(cap, np.int32)
    m, n = demand.shape
    o, st, arrs, keep = _options(m, n_starts, max_rounds, order_seed, orders,
                                 flags)
    tgt = np.zeros((m, n), np.uint8)
    obj = ctypes.c_int64(0)
    _check(lib().pp_plan(n, m, _p(parent), _p(demand), _p(w), _p(f), _p(cap),
                         ctypes.byref(o), _p(tgt), ctypes.byref(obj),
                         ctypes.byref(st)))
    del keep
    return _plan_from(st, arrs, tgt, obj.value)


@dataclass
class Replan:
    target: np.ndarray          # uint8 [m][n]: the placement to use
    proposal: np.ndarray        # uint8 [m][n]: the re-optimized plan
    adopt: bool
    incumbent_objective: int
    proposal_objective: int
    materialization_cost: int
    plan: Plan                  # the proposal's planner statistics


def pp_replan(parent, demand, recompute_cost, fetch_cost, cap, incumbent,
              horizon, *, n_starts=8, max_rounds=0, order_seed=0, orders=None,
              flags=0) -> Replan:
    """Epoch re-planning (see pp_replan in include/prefixplace.h)."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    cap = _c(cap, np.int32)
    inc = _c(incumbent, np.uint8)
    m, n = demand.shape
    if inc.shape != (m, n):
        raise ValueError(f"incumbent shape {inc.shape} != {(m, n)}")
    o, st, arrs, keep = _options(m, n_starts, max_rounds, order_seed, orders,
                                 flags)
    tgt = np.zeros((m, n), np.uint8)
    prop = np.zeros((m, n), np.uint8)
    info = pp_replan_info()
    _check(lib().pp_replan(n, m, _p(parent), _p(demand), _p(w), _p(f), _p(cap),
                           _p(inc), int(horizon), ctypes.byref(o), _p(tgt),
                           _p(prop), ctypes.byref(info), ctypes.byref(st)))
    del keep
    return Replan(target=tgt, proposal=prop, adopt=bool(info.adopt),
                  incumbent_objective=int(info.incumbent_objective),
                  proposal_objective=int(info.proposal_objective),
                  materialization_cost=int(info.materialization_cost),
                  plan=_plan_from(st, arrs, prop, info.proposal_objective))


def _options_f64(m, n_starts, max_rounds, order_seed, orders, flags):
    o, _, _, keep = _options(m, n_starts, max_rounds, order_seed, orders, flags)
    S = pp_num_starts(m, n_starts)
    st = pp_stats_f64()
    arrs = dict(start_objective=np.zeros(S, np.float64),
                start_sweeps=np.zeros(S, np.int32),
                start_accepts=np.zeros(S, np.int32),
                standalone=np.zeros(m, np.float64),
                orders=np.zeros((S, m), np.int32))
    for k, v in arrs.items():
        setattr(st, k, v.ctypes.data)
    return o, st, arrs, keep


def _plan_f64_from(st, arrs, target, objective):
    return Plan(target=target, objective=float(objective), best_start=st.best_start,
                n_starts=st.n_starts, updates=st.updates, dp_cells=st.dp_cells,
                dp_kernel_ms=st.dp_kernel_ms, dp_launches=st.dp_launches,
                safeguards_run=bool(st.safeguards_run),
                safeguard_objective=tuple(float(x) for x in st.safeguard_objective),
                dp_cells_executed=st.dp_cells_executed,
                dp_lane_cells=st.dp_lane_cells, dp_fmax=bool(st.dp_fmax),
                dp_restarts=st.dp_restarts, **arrs)


def pp_plan_f64(parent, demand, recompute_cost, fetch_cost, cap, *, epsilon=0.0,
                n_starts=8, max_rounds=0, order_seed=0, orders=None, flags=0) -> Plan:
    """Real-valued host-array planner (see pp_plan_f64 in
    include/prefixplace.h); objectives are floats."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.float64)
    w = _c(recompute_cost, np.float64)
    f = _c(fetch_cost, np.float64)
    cap = _c(cap, np.int32)
    m, n = demand.shape
    o, st, arrs, keep = _options_f64(m, n_starts, max_rounds, order_seed, orders,
                                     flags)
    tgt = np.zeros((m, n), np.uint8)
    obj = ctypes.c_double(0.0)
    _check(lib().pp_plan_f64(n, m, _p(parent), _p(demand), _p(w), _p(f), _p(cap),
                             float(epsilon), ctypes.byref(o), _p(tgt),
                             ctypes.byref(obj), ctypes.byref(st)))
    del keep
    return _plan_f64_from(st, arrs, tgt, obj.value)


def pp_replan_f64(parent, demand, recompute_cost, fetch_cost, cap, incumbent,
                  horizon, *, epsilon=0.0, n_starts=8, max_rounds=0, order_seed=0,
                  orders=None, flags=0) -> Replan:
    """Real-valued epoch re-planning (see pp_replan_f64 in
    include/prefixplace.h)."""
    parent = _c(parent, np.int32)
    demand = _c(demand, np.float64)
    w = _c(recompute_cost, np.float64)
    f = _c(fetch_cost, np.float64)
    cap = _c(cap, np.int32)
    inc = _c(incumbent, np.uint8)
    m, n = demand.shape
    if inc.shape != (m, n):
        raise ValueError(f"incumbent shape {inc.shape} != {(m, n)}")
    o, st, arrs, keep = _options_f64(m, n_starts, max_rounds, order_seed, orders,
                                     flags)
    tgt = np.zeros((m, n), np.uint8)
    prop = np.zeros((m, n), np.uint8)
    info = pp_replan_info_f64()
    _check(lib().pp_replan_f64(n, m, _p(parent), _p(demand), _p(w), _p(f),
                               _p(cap), _p(inc), float(horizon), float(epsilon),
                               ctypes.byref(o), _p(tgt), _p(prop),
                               ctypes.byref(info), ctypes.byref(st)))
    del keep
    return Replan(target=tgt, proposal=prop, adopt=bool(info.adopt),
                  incumbent_objective=float(info.incumbent_objective),
                  proposal_objective=float(info.proposal_objective),
                  materialization_cost=float(info.materialization_cost),
                  plan=_plan_f64_from(st, arrs, prop, info.proposal_objective))


def pp_rooted_dp_f64(parent, profit, k):
    parent = _c(parent, np.int32)
    profit = _c(profit, np.float64)
    n = parent.shape[0]
    sel = np.zeros(n, np.uint8)
    val = ctypes.c_double(0.0)
    _check(lib().pp_rooted_dp_f64(n, _p(parent), _p(profit), int(k), _p(sel),
                                  ctypes.byref(val)))
    return sel, val.value


def pp_rooted_dp(parent, profit, k):
    parent = _c(parent, np.int32)
    profit = _c(profit, np.int64)
    n = parent.shape[0]
    sel = np.zeros(n, np.uint8)
    val = ctypes.c_int64(0)
    _check(lib().pp_rooted_dp(n, _p(parent), _p(profit), int(k), _p(sel),
                              ctypes.byref(val)))
    return sel, val.value


def pp_marginal(demand, recompute_cost, fetch_cost, target, h):
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    target = _c(target, np.uint8)
    m, n = demand.shape
    prof = np.zeros(n, np.int64)
    g = ctypes.c_int64(0)
    _check(lib().pp_marginal(n, m, _p(demand), _p(w), _p(f), _p(target),
                             int(h), _p(prof), ctypes.byref(g)))
    return prof, g.value


def pp_objective(demand, recompute_cost, fetch_cost, target) -> int:
    demand = _c(demand, np.int64)
    w = _c(recompute_cost, np.int64)
    f = _c(fetch_cost, np.int64)
    target = _c(target, np.uint8)
    m, n = demand.shape
    out = ctypes.c_int64(0)
    _check(lib().pp_objective(n, m, _p(demand), _p(w), _p(f), _p(target),
                              ctypes.byref(out)))
    return out.value


def pp_objective_device_noalloc(demand_dev, recompute_dev, fetch_dev, target_dev,
                                stream=None) -> int:
    """F_pair(T) on torch device tensors (int64 [m][n], int64 [m][n], int64
    [m][m][n], uint8 [m][n]) through the allocation-free entry point (see
    include/prefixplace.h)."""
    import torch

    for t, dt in ((demand_dev, torch.int64), (recompute_dev, torch.int64),
                  (fetch_dev, torch.int64), (target_dev, torch.uint8)):
        if not t.is_cuda or t.dtype != dt or not t.is_contiguous():
            raise ValueError("device tensors must be contiguous, on the GPU, "
                             "with the documented dtypes")
    m, n = demand_dev.shape
    if tuple(fetch_dev.shape) != (m, m, n) or tuple(target_dev.shape) != (m, n) \
            or tuple(recompute_dev.shape) != (m, n):
        raise ValueError("shape mismatch")
    s = stream if stream is not None else torch.cuda.current_stream()
    out = ctypes.c_int64(0)
    _check(lib().pp_objective_device_noalloc(
        n, m, demand_dev.data_ptr(), recompute_dev.data_ptr(), fetch_dev.data_ptr(),
        target_dev.data_ptr(), ctypes.byref(out), ctypes.c_void_p(s.cuda_stream)))
    return out.value


def pp_orders(m, n_starts, order_seed, standalone):
    st = _c(standalone, np.int64)
    S = pp_num_starts(m, n_starts)
    out = np.zeros((S, m), np.int32)
    _check(lib().pp_orders(m, n_starts, int(order_seed) & (2 ** 64 - 1),
                           _p(st), _p(out)))
    return out


def pp_sweep_layout(parent, cells):
    """Per-step metadata of the DP sweep for a tree (host only)."""
    parent = _c(parent, np.int32)
    n = parent.shape[0]
    ns, sl = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().pp_sweep_layout(n, _p(parent), int(cells), None,
                                 ctypes.byref(ns), ctypes.byref(sl)))
    meta = np.zeros((ns.value, 4), np.uint32)
    _check(lib().pp_sweep_layout(n, _p(parent), int(cells), _p(meta),
                                 ctypes.byref(ns), ctypes.byref(sl)))
    return meta, sl.value


def pp_sweep_spills(parent):
    """Spill schedule of the DP sweep for a deep tree (host only): returns
    (nspill, out lists, in lists), each list one int32 [k][2] array of
    (LDS slot, spill index) per sweep batch."""
    parent = _c(parent, np.int32)
    n = parent.shape[0]
    nb, ns, no, ni = (ctypes.c_int32(0) for _ in range(4))
    _check(lib().pp_sweep_spills(n, _p(parent), ctypes.byref(nb), ctypes.byref(ns),
                                 ctypes.byref(no), ctypes.byref(ni), None, None, None, None))
    out_off = np.zeros(nb.value + 1, np.int32)
    in_off = np.zeros(nb.value + 1, np.int32)
    outs = np.zeros((max(no.value, 1), 2), np.int32)
    ins = np.zeros((max(ni.value, 1), 2), np.int32)
    _check(lib().pp_sweep_spills(n, _p(parent), ctypes.byref(nb), ctypes.byref(ns),
                                 ctypes.byref(no), ctypes.byref(ni), _p(out_off), _p(outs),
                                 _p(in_off), _p(ins)))
    per_out = [outs[out_off[b]:out_off[b + 1]] for b in range(nb.value)]
    per_in = [ins[in_off[b]:in_off[b + 1]] for b in range(nb.value)]
    return ns.value, per_out, per_in


PP_BT_END = 0x7FFFFFFF


def pp_backtrack_table(parent):
    """The backtrack's per-row skip table of a tree, [rows][4] uint32
    (host only; see pp_backtrack_table in include/prefixplace.h)."""
    parent = _c(parent, np.int32)
    n = parent.shape[0]
    rows = ctypes.c_int64(0)
    _check(lib().pp_backtrack_table(n, _p(parent), None, ctypes.byref(rows)))
    table = np.zeros((rows.value, 4), np.uint32)
    _check(lib().pp_backtrack_table(n, _p(parent), _p(table), ctypes.byref(rows)))
    return table


class Context:
    """A reusable GPU context (pp_ctx) for device-resident planning."""

    def __init__(self, device: int = 0):
        self._h = _P()
        _check(lib().pp_ctx_create(ctypes.byref(self._h), int(device)))

    def close(self):
        if self._h:
            lib().pp_ctx_destroy(self._h)
            self._h = _P()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def pp_plan_f64_device(self, parent, demand_dev, recompute_dev, fetch_dev,
                           cap, target_dev, *, epsilon=0.0, n_starts=8,
                           max_rounds=0, order_seed=0, orders=None, flags=0,
                           stream=None) -> Plan:
        """Real-valued plan on torch device tensors (float64 [m][n],
        float64 [m][n], float64 [m][m][n]); writes uint8 [m][n] into
        `target_dev`."""
        import torch

        for t, dt in ((demand_dev, torch.float64), (recompute_dev, torch.float64),
                      (fetch_dev, torch.float64), (target_dev, torch.uint8)):
            if not t.is_cuda or t.dtype != dt or not t.is_contiguous():
                raise ValueError("device tensors must be contiguous, on the "
                                 "GPU, with the documented dtypes")
        parent = _c(parent, np.int32)
        cap = _c(cap, np.int32)
        m, n = demand_dev.shape
        if tuple(fetch_dev.shape) != (m, m, n) or tuple(target_dev.shape) != (m, n) \
                or tuple(recompute_dev.shape) != (m, n) or parent.shape[0] != n \
                or cap.shape[0] != m:
            raise ValueError("shape mismatch")
        o, st, arrs, keep = _options_f64(m, n_starts, max_rounds, order_seed,
                                         orders, flags)
        obj = ctypes.c_double(0.0)
        s = stream if stream is not None else torch.cuda.current_stream()
        _check(lib().pp_plan_f64_device(
            self._h, n, m, _p(parent), demand_dev.data_ptr(),
            recompute_dev.data_ptr(), fetch_dev.data_ptr(), _p(cap),
            float(epsilon), ctypes.byref(o), target_dev.data_ptr(),
            ctypes.byref(obj), ctypes.byref(st), ctypes.c_void_p(s.cuda_stream)))
        del keep
        return _plan_f64_from(st, arrs, target_dev, obj.value)

    def pp_plan_device(self, parent, demand_dev, recompute_dev, fetch_dev, cap,
                       target_dev, *, n_starts=8, max_rounds=0, order_seed=0,
                       orders=None, flags=0, stream=None) -> Plan:
        """Plan on torch device tensors (int64 [m][n], int64 [m][n],
        int64 [m][m][n]); writes uint8 [m][n] into `target_dev`."""
        import torch

        for t, dt in ((demand_dev, torch.int64), (recompute_dev, torch.int64),
                      (fetch_dev, torch.int64), (target_dev, torch.uint8)):
            if not t.is_cuda or t.dtype != dt or not t.is_contiguous():
                raise ValueError("device tensors must be contiguous, on the "
                                 "GPU, with the documented dtypes")
        parent = _c(parent, np.int32)
        cap = _c(cap, np.int32)
        m, n = demand_dev.shape
        if tuple(fetch_dev.shape) != (m, m, n) or tuple(target_dev.shape) != (m, n) \
                or tuple(recompute_dev.shape) != (m, n) or parent.shape[0] != n \
                or cap.shape[0] != m:
            raise ValueError("shape mismatch")
        o, st, arrs, keep = _options(m, n_starts, max_rounds, order_seed,
                                     orders, flags)
        obj = ctypes.c_int64(0)
        s = stream if stream is not None else torch.cuda.current_stream()
        _check(lib().pp_plan_device(
            self._h, n, m, _p(parent), demand_dev.data_ptr(),
            recompute_dev.data_ptr(), fetch_dev.data_ptr(), _p(cap),
            ctypes.byref(o), target_dev.data_ptr(), ctypes.byref(obj),
            ctypes.byref(st), ctypes.c_void_p(s.cuda_stream)))
        del keep
        return _plan_from(st, arrs, target_dev, obj.value)
