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


def test_cluster_order_key_worked_by_hand():
    # The order after propagation sorts by (label, -degree, id), the degree counting a row's entries other than
    # its self-loop.  Six nodes in two clusters, labels given; rows chosen so that each part of the key decides
    # somewhere (worked by hand):
    #   node: 0      1        2      3        4    5
    #   row : {0,2}  {1,3,5}  {0,4}  {0,1,2}  {4}  {1,3}
    #   deg : 1      2        2      3        0    2      (self-loops of 0, 1, 4 not counted)
    #   lab : 5      2        5      2        5    2
    # cluster 2 first: 3 (deg 3), then 1 and 5 (deg 2, by id); cluster 5: 2 (deg 2), 0 (deg 1), 4 (deg 0).
    # Counting self-loops would give [1, 3, 5, 0, 2, 4]; an ascending degree [1, 5, 3, 4, 0, 2]; no label
    # [3, 1, 2, 5, 0, 4]; ties by descending id [3, 5, 1, 2, 0, 4].
    rows = [[0, 2], [1, 3, 5], [0, 4], [0, 1, 2], [4], [1, 3]]
    rowptr = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int64)
    col = np.concatenate(rows).astype(np.int32)
    labels = np.array([5, 2, 5, 2, 5, 2])
    perm, iperm = R.cluster_order(rowptr, col, labels)
    assert perm.tolist() == [3, 1, 5, 2, 0, 4]
    assert iperm.tolist() == [4, 1, 3, 0, 5, 2]


def test_reorder_orders_unequal_degree_clusters_by_degree():
    # End to end through propagation: two disjoint graphs, a 5-clique with two pendant nodes on member a and
    # one on member b, and a triangle with one pendant.  Each component converges to one label (checked), and
    # inside a component the nodes come out by falling degree (self-loops, added by csr_from_pairs, ignored),
    # ties by id.
    rng = np.random.default_rng(8)
    n = 12
    ids = rng.permutation(n)
    k5 = ids[:5]
    pend = ids[5:8]
    tri = ids[8:11]
    tri_pend = ids[11]
    u, v = [], []
    for a in range(5):
        for b in range(a + 1, 5):
            u.append(k5[a]); v.append(k5[b])
    u += [k5[0], k5[0], k5[1]]; v += [pend[0], pend[1], pend[2]]
    u += [tri[0], tri[0], tri[1], tri[2]]; v += [tri[1], tri[2], tri[2], tri_pend]
    rowptr, col = csr_from_pairs(n, u, v)
    perm, iperm, lab = R.reorder(rowptr, col)
    comp1 = set(k5.tolist()) | set(pend.tolist())
    comp2 = set(tri.tolist()) | {int(tri_pend)}
    assert len({int(lab[x]) for x in comp1}) == 1 and len({int(lab[x]) for x in comp2}) == 1
    deg = {int(x): 0 for x in range(n)}
    for a, b in zip(u, v):
        deg[int(a)] += 1
        deg[int(b)] += 1
    first, second = (comp1, comp2) if lab[k5[0]] < lab[tri[0]] else (comp2, comp1)
    expect = sorted(first, key=lambda x: (-deg[x], x)) + sorted(second, key=lambda x: (-deg[x], x))
    assert perm.tolist() == expect
