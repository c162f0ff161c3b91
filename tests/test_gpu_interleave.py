"""The interleave decision on the GPU (§3.2, conditions C1-C3) against the oracle: every field of the report
and the first search's depths, on textbook graphs, random graphs, and the workloads at full size."""

import numpy as np
import pytest
import torch

from oracle import interleave as OI
from synth import csr_from_pairs, make_workload
from tests.helpers import dev_csr

pytestmark = pytest.mark.gpu


def check(gt, rowptr, col, L):
    ref = OI.interleave_report(rowptr, col, L)
    rp, cl = dev_csr(rowptr, col)
    got, lev = gt.interleave_check(rp, cl, L, want_levels=True)
    torch.cuda.synchronize()
    for key, val in ref.items():
        assert got[key] == val, (key, got[key], val, L)
    if len(rowptr) > 1:
        assert np.array_equal(lev.cpu().numpy(), OI.bfs_levels(rowptr, col, 0, L + 1))
    return got


def graph(n, pairs, loops=True):
    u = np.array([p[0] for p in pairs], np.int64)
    v = np.array([p[1] for p in pairs], np.int64)
    return csr_from_pairs(n, u, v, symmetric=True, self_loops=loops)


def test_textbook_graphs(gt):
    cases = [
        graph(1, []), graph(2, []), graph(2, [(0, 1)]),
        graph(7, [(i, j) for i in range(7) for j in range(i + 1, 7)]),            # complete
        graph(7, [(i, j) for i in range(7) for j in range(i + 1, 7)], loops=False),
        graph(9, [(i, (i + 1) % 9) for i in range(9)]),                          # cycle
        graph(4, [(i, (i + 1) % 4) for i in range(4)]),
        graph(12, [(i, i + 1) for i in range(11)]),                              # path
        graph(6, [(5, i) for i in range(5)]),                                    # star, root a leaf
        graph(6, [(0, 1), (1, 2), (3, 4), (4, 5)]),                              # two components
    ]
    for rp, cl in cases:
        for L in (0, 1, 2, 3, 5, 8, 11, 22, 40):
            check(gt, rp, cl, L)


@pytest.mark.parametrize("seed", range(20))
def test_random_graphs(gt, seed):
    rng = np.random.default_rng(200 + seed)
    n = int(rng.integers(2, 400))
    m = int(rng.integers(0, 3 * n))
    rp, cl = csr_from_pairs(n, rng.integers(0, n, m), rng.integers(0, n, m), symmetric=True,
                            self_loops=bool(seed % 4))
    for L in (1, 3, 6, 12, 30):
        check(gt, rp, cl, L)


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "b1"])
def test_workloads_full_size(gt, name):
    g = make_workload(name).graph
    for L in (2, 4, 8, 12):
        got = check(gt, g.rowptr, g.col, L)
        print(name, L, got, flush=True)
