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
