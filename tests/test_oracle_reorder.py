"""Pins of the reorder oracle (cluster reordering of §3.3, label-propagation reading).

* SplitMix64 output function against the published reference outputs;
* one sweep worked by hand on a star;
* structural facts: bijection, identity on an edgeless graph, each clique of a
  disjoint union of cliques contiguous and single-labelled, fixed-point
  property at convergence (checked by plain per-node counting);
* quality: on a planted block model the order packs about as many edges into
  dense tiles as the planted block order does.
"""

import collections
import os

import numpy as np

from oracle import plan as P
from oracle import reorder as R
from synth import csr_from_pairs, make_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64_seed0.txt")


def test_splitmix64_reference_outputs():
    vals = [int(line, 16) for line in open(GOLDEN) if line.strip() and not line.startswith("#")]
    G = 0x9E3779B97F4A7C15
    got = [int(R.mix64(np.uint64((k * G) % (1 << 64)))) for k in range(1, len(vals) + 1)]
    assert got == vals


def test_star_first_sweep_by_hand():
    # center 0, leaves 1..3 (self-loops present but ignored)
    rowptr, col = csr_from_pairs(4, [0, 0, 0], [1, 2, 3])
    n, r, c = R._offdiag_edges(rowptr, col)
    lab = np.arange(4)
    cand, new = R.lp_sweep(n, r, c, lab, 0, seed=0)
    # every leaf sees only label 0 (its own label is not among it) -> 0
    assert list(cand[1:]) == [0, 0, 0]
    # the center sees {1,2,3} once each; its own label 0 is absent -> smallest (h_0(l), l)
    k = (0 + 1 * 0x9E3779B97F4A7C15) % (1 << 64)
    pri = {l: int(R.mix64(np.uint64(l ^ k))) for l in (1, 2, 3)}
    assert cand[0] == min((pri[l], l) for l in (1, 2, 3))[1]
    act = [(int(R.mix64(np.uint64(v ^ k ^ 0xD6E8FEB86659FD93))) >> 61) != 0 for v in range(4)]
    assert list(new) == [int(cand[v]) if act[v] else v for v in range(4)]


def test_bijection_on_workload_graph():
    g = make_workload("c1", 0.25).graph
    perm, iperm, _ = R.reorder(g.rowptr, g.col)
    assert sorted(perm.tolist()) == list(range(g.n))
    np.testing.assert_array_equal(iperm[perm], np.arange(g.n))


def test_edgeless_graph_gives_identity():
    rowptr, col = csr_from_pairs(50, [], [])  # self-loops only
    perm, iperm, lab = R.reorder(rowptr, col)
    np.testing.assert_array_equal(perm, np.arange(50))
    np.testing.assert_array_equal(lab, np.arange(50))


def test_disjoint_cliques_come_out_contiguous():
    rng = np.random.default_rng(3)
    sizes = [5, 9, 4, 12, 7, 6]
    n = sum(sizes)
    ids = rng.permutation(n)
    u, v = [], []
    start = 0
    groups = []
    for s in sizes:
        members = ids[start:start + s]
        groups.append(set(members.tolist()))
        for a in range(s):
            for b in range(a + 1, s):
                u.append(members[a])
                v.append(members[b])
        start += s
    rowptr, col = csr_from_pairs(n, u, v)
    perm, iperm, lab = R.reorder(rowptr, col)
    for grp in groups:
        pos = sorted(iperm[list(grp)])
        assert pos[-1] - pos[0] == len(grp) - 1
        assert len({int(lab[x]) for x in grp}) == 1


def test_converged_labels_are_a_fixed_point():
    g = make_workload("c5", 0.1).graph
    lab, done = R.lp_labels(g.rowptr, g.col, iters=200)
    assert done < 200
    for v in range(g.n):
        nb = [int(u) for u in g.col[g.rowptr[v]:g.rowptr[v + 1]] if u != v]
        if not nb:
            continue
        cnt = collections.Counter(int(lab[u]) for u in nb)
        assert cnt[int(lab[v])] == max(cnt.values())


def _dense_edge_share(g, perm, iperm, T=128, tau=0.01):
    rp, c = P.permute_csr(g.rowptr, g.col, perm, iperm)
    pl = P.build_tiles(rp, c, T, P.tau_to_ppm(tau))
    return 1.0 - len(pl["sp_col"]) / g.nnz


def test_recovers_planted_blocks_about_as_well_as_planted_order():
    g = make_workload("c4", 0.05).graph
    planted = np.lexsort((np.arange(g.n), g.block))
    ip = np.empty(g.n, np.int64)
    ip[planted] = np.arange(g.n)
    perm, iperm, _ = R.reorder(g.rowptr, g.col)
    ours = _dense_edge_share(g, perm, iperm)
    ref = _dense_edge_share(g, planted, ip)
    assert ref > 0.8
    assert ours >= 0.95 * ref
