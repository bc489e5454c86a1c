"""Checks of the seeded input generator (no planner arithmetic involved)."""

import numpy as np
import pytest

from paper_2608_01655_amd import workloads as W


def test_chunk_fetch_constants():
    """36,864 B/token x 512 tokens = 18,874,368 B ("18.9 MB", Sec. I); at
    1.5 Gb/s that is about 100.7 ms (Fig. 1 caption)."""
    assert W.CHUNK_BYTES == 18_874_368
    assert int(W.fetch_us_for_gbps(1.5)) == 100_663
    assert abs(int(W.fetch_us_for_gbps(1.5)) - 100_700) < 100


@pytest.mark.parametrize("name", ["tiny", "tree2k", "rag10k"])
def test_small_workloads_shape(name):
    inst = W.make_workload(name)
    n, m = inst.n, inst.m
    assert inst.demand.shape == (m, n)
    assert inst.fetch_cost.shape == (m, m, n)
    # preorder labels: every parent precedes its child
    assert np.all(inst.parent[1:] < np.arange(1, n))
    assert inst.parent[0] == -1
    # demand of a node = sum of its children's plus its own leaf requests
    child_sum = np.zeros_like(inst.demand)
    for v in range(1, n):
        child_sum[:, inst.parent[v]] += inst.demand[:, v]
    has_child = np.zeros(n, bool)
    has_child[inst.parent[1:]] = True
    assert np.all(inst.demand[:, has_child] == child_sum[:, has_child])
    assert np.all(inst.demand >= 0) and np.all(inst.recompute_cost > 0)
    for h in range(m):
        assert np.all(inst.fetch_cost[h, h] == 0)


def test_workload_totals_and_depths():
    for name, total, dmax in (("tiny", 10_000, 8), ("tree2k", 10 ** 6, 12),
                              ("rag10k", 10 ** 7, 7)):
        inst = W.make_workload(name)
        assert int(inst.demand[:, 0].sum()) == total
        assert int(inst.depth.max()) <= dmax
    tiny = W.make_workload("tiny")
    assert tiny.n == 200 and tiny.m == 2
    assert np.all(tiny.fetch_cost[0, 1] == 100_700)
    # h = [1.0, 2.5], a = 20,000, b = 6,000
    d = tiny.depth.astype(np.int64)
    assert np.array_equal(tiny.recompute_cost[0], 20_000 + 6_000 * d)
    assert np.array_equal(tiny.recompute_cost[1], (25 * (20_000 + 6_000 * d)) // 10)


def test_generator_is_deterministic():
    a = W.make_workload("tree2k")
    b = W.make_workload("tree2k")
    assert a.checksum() == b.checksum()


def test_routing_shift_and_popularity_perturbation():
    inst = W.make_workload("tree2k")
    lam = inst.demand
    full = W.shift_routing(inst.parent, lam, 1, 1)
    np.testing.assert_array_equal(full, np.roll(lam, 1, axis=0))
    none = W.shift_routing(inst.parent, lam, 0, 4)
    np.testing.assert_array_equal(none, lam)
    for num in (1, 2):
        part = W.shift_routing(inst.parent, lam, num, 4)
        # requests only move between workers: per-node totals are kept
        np.testing.assert_array_equal(part.sum(axis=0), lam.sum(axis=0))
        assert part.min() >= 0
    rng = np.random.default_rng(3)
    pert = W.perturb_popularity(inst.parent, lam, 0.5, rng)
    assert pert.min() >= 0 and pert.shape == lam.shape
    # still aggregated along prefix paths: a node covers its children
    for v in range(1, inst.n):
        p = inst.parent[v]
        if p >= 0:
            assert np.all(pert[:, p] >= pert[:, v])
    zero = W.perturb_popularity(inst.parent, lam, 0.0, rng)
    np.testing.assert_array_equal(zero, lam)


def test_runtime_instances_share_the_tree():
    """The n = 10,000, k = 128 runtime configurations: one RAG-shaped tree
    for M = 4, 8 and 16, demand aggregated along prefix paths with the same
    total, the paper's default start set."""
    insts = [W.runtime_instance(m) for m in (4, 8, 16)]
    for inst, m in zip(insts, (4, 8, 16)):
        assert inst.n == 10_000 and inst.m == m
        np.testing.assert_array_equal(inst.parent, insts[0].parent)
        assert inst.cap.tolist() == [128] * m and inst.n_starts == 0
        assert int(inst.demand[:, 0].sum()) == 10 ** 7
        assert inst.fetch_cost.shape == (m, m, inst.n)
        for v in range(1, inst.n):
            p = inst.parent[v]
            if p >= 0:
                assert np.all(inst.demand[:, p] >= inst.demand[:, v])
