"""CPU check of the backtrack's skip table (no GPU).

Theorem 1's walk from (1, k') moves to row i+1 on a take and to next(i) on a
skip.  The library's walk advances per take: for each row q it uses the
rows of q, next(q), next(next(q)), ... inside q's 32-row window (a mask),
the first such row past the window (the exit) and that row's own mask.
This test rebuilds the table from the definition -- canonical preorder,
subtree sizes, the skip sequence followed row by row -- and requires the
library's table to match it word for word, padding included.
"""

import numpy as np
import pytest

from paper_2608_01655_amd import binding as B
from paper_2608_01655_amd import workloads as W
from tests import bruteforce as bf

END = B.PP_BT_END


def table_by_definition(parent):
    n = len(parent)
    order = bf.canonical_preorder(parent)
    pos = {v: i for i, v in enumerate(order)}
    size = [1] * n
    for i in range(n - 1, -1, -1):
        p = int(parent[order[i]])
        if p >= 0:
            size[pos[p]] += size[i]
    nxt = [i + size[i] for i in range(n)]
    rows = (n + 511) // 512 * 512 + 512
    out = np.zeros((rows, 4), np.uint32)
    out[n:, 1] = END

    def mask_exit(q):
        bound = min((q // 32 + 1) * 32, n)
        m, r = 0, q
        while r < bound:
            m |= 1 << (r % 32)
            r = nxt[r]
        return m, (r if r < n else END)

    for q in range(n):
        m, e = mask_exit(q)
        out[q, 0] = m
        out[q, 1] = e
        out[q, 2] = mask_exit(e)[0] if e != END else 0
    return out


@pytest.mark.parametrize("seed", range(12))
def test_backtrack_table_random(seed):
    rng = np.random.default_rng(9000 + seed)
    n = int(rng.choice([1, 31, 32, 33, 511, 512, 513, 1100, 1536]))
    parent = W.random_forest(n, rng, p_root=float(rng.choice([0.0, 0.02, 0.3])))
    np.testing.assert_array_equal(B.pp_backtrack_table(parent),
                                  table_by_definition(parent))


def test_backtrack_table_shapes():
    """A path (every skip leaves the tree), a star, a forest of singletons
    and a comb whose leaves are skip targets deep in the preorder."""
    n = 700
    path = np.arange(-1, n - 1, dtype=np.int32)
    star = np.array([-1] + [0] * (n - 1), np.int32)
    flat = np.full(n, -1, np.int32)
    # spine 0..199 with a leaf 200+d under spine node d (the sweep's LDS
    # slots bound the depth of pending skip targets)
    comb = np.array([-1] + list(range(0, 199)) + list(range(0, 200)), np.int32)
    for parent in (path, star, flat, comb):
        np.testing.assert_array_equal(B.pp_backtrack_table(parent),
                                      table_by_definition(parent))


def test_backtrack_table_rejects_bad_trees():
    with pytest.raises(B.PPError):
        B.pp_backtrack_table(np.array([1, 0], np.int32))  # a cycle
