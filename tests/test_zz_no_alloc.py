"""The allocation-free objective entry point against pp_objective.

pp_objective_device_noalloc evaluates F_pair(T) (Eq. 6) with no allocation,
its partial sums in the library's per-GPU scratch array.  Two calls in a
row, the second on a smaller input, must each equal pp_objective bit for
bit (and the oracle's value), so that nothing left in the scratch by the
first call leaks into the second.
"""

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _say_case(request):
    print(f"\n[case] {request.node.name}", flush=True)
    yield


def _dev(inst, target):
    import torch

    d = torch.device("cuda:0")
    return (torch.from_numpy(np.ascontiguousarray(inst.demand)).to(d),
            torch.from_numpy(np.ascontiguousarray(inst.recompute_cost)).to(d),
            torch.from_numpy(np.ascontiguousarray(inst.fetch_cost)).to(d),
            torch.from_numpy(np.ascontiguousarray(target)).to(d))


def _random_target(rng, m, n):
    t = (rng.random((m, n)) < 0.3).astype(np.uint8)
    t[t != 0] = rng.integers(1, 256, size=int(t.sum()), dtype=np.uint8)  # any nonzero byte holds
    return t


@pytest.mark.parametrize("seed", range(6))
def test_two_calls_second_smaller(oracle_mod, seed):
    import torch

    rng = np.random.default_rng(4400 + seed)
    big = W.random_instance(int(rng.integers(2000, 6000)), int(rng.integers(3, 9)),
                            rng, kmax=50, source_dependent=True)
    small = W.random_instance(int(rng.integers(1, 300)), int(rng.integers(1, 4)),
                              rng, kmax=10, source_dependent=bool(seed % 2))
    for inst in (big, small):
        tgt = _random_target(rng, inst.m, inst.n)
        got = B.pp_objective_device_noalloc(*_dev(inst, tgt))
        torch.cuda.synchronize()
        ref = B.pp_objective(inst.demand, inst.recompute_cost, inst.fetch_cost, tgt)
        assert got == ref
        assert got == oracle_mod.objective(inst.demand, inst.recompute_cost,
                                           inst.fetch_cost, (tgt != 0).astype(np.uint8))


def test_workload_sizes_then_tiny(oracle_mod):
    """tree50k's 16 x 50,000 inputs (more partial sums than the kernel has
    blocks: a grid-stride loop), then the 200-chunk workload."""
    for name in ("tree50k", "tiny"):
        inst = W.make_workload(name)
        ref = oracle_mod.plan_instance(inst) if name == "tiny" else None
        tgt = ref.target if ref is not None else W.prefix_incumbent(inst.n, inst.cap)
        got = B.pp_objective_device_noalloc(*_dev(inst, tgt))
        assert got == B.pp_objective(inst.demand, inst.recompute_cost,
                                     inst.fetch_cost, tgt)
        if ref is not None:
            assert got == ref.objective


def test_errors_leave_output_and_next_call_clean():
    """A negative cost is reported (PP_E_RANGE) and the following call on
    valid inputs is still exact."""
    rng = np.random.default_rng(5)
    inst = W.random_instance(500, 4, rng, kmax=20, source_dependent=True)
    tgt = _random_target(rng, inst.m, inst.n)
    bad = inst.fetch_cost.copy()
    bad[1, 2, 7] = -1
    import dataclasses

    with pytest.raises(B.PPError) as ei:
        B.pp_objective_device_noalloc(*_dev(dataclasses.replace(inst, fetch_cost=bad), tgt))
    assert ei.value.code == B.PP_E_RANGE
    got = B.pp_objective_device_noalloc(*_dev(inst, tgt))
    assert got == B.pp_objective(inst.demand, inst.recompute_cost, inst.fetch_cost, tgt)
