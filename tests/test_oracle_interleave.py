"""Pins of the interleave-decision oracle (§3.2, conditions C1-C3): textbook graphs with known degrees,
Hamiltonian structure and diameters, and breadth-first depths checked against scipy's shortest paths."""

import numpy as np
import pytest
from scipy.sparse import csr_matrix
from scipy.sparse.csgraph import shortest_path

from oracle import interleave as OI
from synth import csr_from_pairs


def graph(n, pairs, loops=True):
    u = np.array([p[0] for p in pairs], np.int64)
    v = np.array([p[1] for p in pairs], np.int64)
    return csr_from_pairs(n, u, v, symmetric=True, self_loops=loops)


def path(n):
    return graph(n, [(i, i + 1) for i in range(n - 1)])


def test_c1_counts_rows_without_self_loop():
    rp, cl = graph(6, [(0, 1), (2, 3)], loops=False)
    assert OI.interleave_report(rp, cl, 4)["missing_self_loops"] == 6
    rp, cl = graph(6, [(0, 1), (2, 3)])
    r = OI.interleave_report(rp, cl, 4)
    assert r["missing_self_loops"] == 0 and r["c1"] == 1


@pytest.mark.parametrize("n", [3, 4, 7, 10])
def test_dirac_on_complete_and_cycle_graphs(n):
    rp, cl = graph(n, [(i, j) for i in range(n) for j in range(i + 1, n)])  # K_n: min degree n - 1
    r = OI.interleave_report(rp, cl, 8)
    assert r["min_degree"] == n - 1 and r["c2"] == 1
    rp, cl = graph(n, [(i, (i + 1) % n) for i in range(n)])  # C_n: min degree 2, Dirac confirms only n <= 4
    r = OI.interleave_report(rp, cl, 8)
    assert r["min_degree"] == 2 and r["c2"] == (1 if n <= 4 else 0)


def test_small_node_counts():
    assert OI.interleave_report(*graph(1, []), 1)["c2"] == 1
    assert OI.interleave_report(*graph(2, [(0, 1)]), 1)["c2"] == 1
    assert OI.interleave_report(*graph(2, []), 1)["c2"] == 0


def test_c3_on_paths_stars_and_components():
    rp, cl = path(6)  # diameter 5, root 0 is an end: eccentricity 5
    assert OI.interleave_report(rp, cl, 4)["c3"] == 0
    assert OI.interleave_report(rp, cl, 10)["c3"] == 1
    r = OI.interleave_report(rp, cl, 7)  # 5 <= 7 < 10: the double sweep finds 5, undetermined
    assert r["c3"] == -1 and r["ecc_root"] == 5 and r["ecc_far"] == 5
    star = graph(6, [(5, i) for i in range(5)])  # centre 5; root 0 is a leaf: eccentricity 2 = diameter
    r = OI.interleave_report(*star, 2)
    assert r["ecc_root"] == 2 and r["c3"] == -1 and r["ecc_far"] == 2
    assert OI.interleave_report(*star, 4)["c3"] == 1
    assert OI.interleave_report(*star, 1)["c3"] == 0
    two = graph(6, [(0, 1), (1, 2), (3, 4), (4, 5)])
    r = OI.interleave_report(*two, 10)
    assert r["c3"] == 0 and r["reached"] == 3
    assert r["use_sparse"] == 0


def test_use_sparse_needs_all_three():
    rp, cl = graph(5, [(i, j) for i in range(5) for j in range(i + 1, 5)])
    r = OI.interleave_report(rp, cl, 2)
    assert (r["c1"], r["c2"], r["c3"], r["use_sparse"]) == (1, 1, 1, 1)
    rp, cl = graph(5, [(i, j) for i in range(5) for j in range(i + 1, 5)], loops=False)
    assert OI.interleave_report(rp, cl, 2)["use_sparse"] == 0


@pytest.mark.parametrize("seed", range(15))
def test_bfs_and_verdicts_against_shortest_paths(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 60))
    m = int(rng.integers(0, 2 * n))
    rp, cl = csr_from_pairs(n, rng.integers(0, n, m), rng.integers(0, n, m), symmetric=True, self_loops=True)
    D = shortest_path(csr_matrix((np.ones(len(cl)), cl, rp), shape=(n, n)), unweighted=True)
    for cap in (1, 3, 100):
        lev = OI.bfs_levels(rp, cl, 0, cap)
        want = np.where(D[0] <= cap, D[0], -1)
        assert np.array_equal(lev, want.astype(np.int64))
    diam = D.max()
    for L in (1, 2, 4, 8, 16):
        c3 = OI.interleave_report(rp, cl, L)["c3"]
        if c3 == 1:
            assert diam <= L
        elif c3 == 0:
            assert diam > L
