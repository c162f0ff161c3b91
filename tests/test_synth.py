"""The seeded generators produce well-formed inputs of the stated shape."""

import numpy as np
import torch

from synth import bf16_bits, bf16_round, chung_lu_graph, make_workload, sbm_graph
from synth.tensors import bf16_to_f32


def check_csr(g):
    rp, c = g.rowptr, g.col
    assert rp.dtype == np.int64 and c.dtype == np.int32 and rp[0] == 0 and len(rp) == g.n + 1
    assert np.all(np.diff(rp) >= 1)  # self-loops: no empty row
    rows = np.repeat(np.arange(g.n), np.diff(rp))
    key = rows * g.n + c
    assert np.all(np.diff(key) > 0)  # sorted, unique
    assert c.min() >= 0 and c.max() < g.n
    # symmetric
    t = np.sort(c.astype(np.int64) * g.n + rows)
    np.testing.assert_array_equal(t, key)
    # self-loops present
    assert np.isin(np.arange(g.n) * (g.n + 1), key).all()


def test_sbm_shape_and_cross_share():
    g = sbm_graph(np.full(20, 150), 12, 0.1, seed=5)
    check_csr(g)
    rows = np.repeat(np.arange(g.n), np.diff(g.rowptr))
    off = rows != g.col
    cross = (g.block[rows[off]] != g.block[g.col[off]]).mean()
    assert abs(cross - 0.1) < 0.02
    assert abs(off.sum() / g.n - 12) < 0.5


def test_chung_lu_shape():
    g = chung_lu_graph(20000, 2.1, 12, 400, seed=3)
    check_csr(g)
    deg = np.diff(g.rowptr) - 1
    assert 9 < deg.mean() < 12.5
    assert deg.max() > 100


def test_workloads_small_scale():
    for name in ("c1", "c2", "c3", "c4", "c5"):
        w = make_workload(name, 0.02)
        check_csr(w.graph)
        q, k, v, do = w.tensors()
        assert q.shape == (w.graph.n, w.heads, w.dim)
        assert (do is not None) == w.backward
    # same seed, same graph
    a, b = make_workload("c1"), make_workload("c1")
    np.testing.assert_array_equal(a.graph.col, b.graph.col)


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32)
    x[:4] = [1.0 + 2**-8, 1.0 + 3 * 2**-8, -(1.0 + 2**-8), 65504.0]  # ties
    ref = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(bf16_round(x), ref)
    np.testing.assert_array_equal(bf16_to_f32(bf16_bits(x)), ref)


def test_batched_graphs_block_diagonal_connected_with_global_token():
    from synth import batched_graphs

    sizes = np.array([3, 25, 24, 1, 26])
    g = batched_graphs(sizes, 2.2, seed=7, global_token=True)
    n_real = int(sizes.sum())
    assert g.n == n_real + 1
    rp, cl = g.rowptr, g.col
    starts = np.concatenate([[0], np.cumsum(sizes)])
    token = n_real
    # symmetric, sorted, self-loops, token row/column complete
    dense = np.zeros((g.n, g.n), dtype=bool)
    for i in range(g.n):
        row = cl[rp[i]:rp[i + 1]]
        assert np.all(np.diff(row) > 0)
        dense[i, row] = True
    assert np.array_equal(dense, dense.T)
    assert dense.diagonal().all()
    assert dense[token].all() and dense[:, token].all()
    # block-diagonal apart from the token, and every small graph connected
    for a, b in zip(starts[:-1], starts[1:]):
        blk = dense[a:b, a:b]
        outside = dense[a:b, :n_real].copy()
        outside[:, a:b] = False
        assert not outside.any()
        seen = {0}
        frontier = [0]
        while frontier:
            u = frontier.pop()
            for v in np.nonzero(blk[u])[0]:
                if v not in seen:
                    seen.add(int(v))
                    frontier.append(int(v))
        assert len(seen) == b - a


def test_batched_workloads_shapes():
    from synth import make_workload

    w = make_workload("b1", 0.01)
    deg = np.diff(w.graph.rowptr)
    assert deg.max() == w.graph.n  # the global token attends to every node, itself included
    assert w.graph.info["graphs"] == 400
    w2 = make_workload("b2", 0.05)
    assert w2.graph.info["global_token"] and w2.graph.n > 3 * 2
