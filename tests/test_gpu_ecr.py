"""The lossy cluster reformation on the GPU (§3.4, cluster sparsity and transfer strategy) against the oracle,
bit for bit: random small graphs over k, d_b and thresholds, clipped and empty clusters, the Auto Tuner's
ladder on a clustered graph after the GPU reorder, the full-size power-law and block-model workloads, and the
exact attention path run on the rewritten graph."""

import sys

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import ecr as OE
from synth import csr_from_pairs, make_workload
from tests.helpers import assert_close, dev_csr, dev_feat, host

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check(gt, rowptr, col, k, d_b, num, den, progress=None):
    rp_ref, cl_ref, info = OE.ecr_compact(rowptr, col, k, d_b, num, den, progress=progress)
    rp, cl = dev_csr(rowptr, col)
    rp2, cl2, moved = gt.ecr_compact(rp, cl, k, d_b, num, den)
    torch.cuda.synchronize()
    assert np.array_equal(rp2.cpu().numpy(), rp_ref), (k, d_b, num, den)
    assert np.array_equal(cl2.cpu().numpy(), cl_ref), (k, d_b, num, den)
    assert moved == int(info["transfer"].sum())
    return rp2, cl2, info


@pytest.mark.parametrize("seed", range(24))
def test_random_small_graphs(gt, seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(1, 200))
    m = int(rng.integers(0, 4 * n + 1))
    u, v = rng.integers(0, n, m), rng.integers(0, n, m)
    rowptr, col = csr_from_pairs(n, u, v, symmetric=bool(seed % 2), self_loops=bool(seed % 3))
    k = int(rng.integers(1, 12))
    d_b = int(rng.integers(1, 9))
    num, den = int(rng.integers(0, 9)), int(rng.integers(1, 9))
    check(gt, rowptr, col, k, d_b, num, den)


def test_edge_cases(gt):
    # a single node, no edges; a graph with no edges; more clusters than nodes; sub-blocks wider than a cluster
    for n, pairs in ((1, []), (10, []), (5, [(0, 1), (1, 2), (3, 4)]), (37, [(i, (7 * i + 3) % 37) for i in range(37)])):
        u = np.array([p[0] for p in pairs], np.int64)
        v = np.array([p[1] for p in pairs], np.int64)
        rowptr, col = csr_from_pairs(n, u, v, symmetric=True, self_loops=True)
        for k, d_b in ((1, 1), (8, 3), (64, 2), (3, 256)):
            for num, den in ((0, 1), (1, 1), (1, 3)):
                check(gt, rowptr, col, k, d_b, num, den)


def test_ladder_on_clustered_graph(gt):
    w = make_workload("c5", 0.05)
    g = w.graph
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2 = gt.permute_csr(rp, cl, perm, iperm)
    r, c = rp2.cpu().numpy(), cl2.cpu().numpy()
    tuner = gt.AutoTuner(g.n, g.nnz, 10)
    rungs = [(int(tuner.c.num[i]), int(tuner.c.den[i])) for i in range(gt.GT_AUTOTUNER_RUNGS)]
    seen = []
    for num, den in rungs:
        _, cl3, info = check(gt, r, c, 8, 16, num, den)
        seen.append(int(info["transfer"].sum()))
        say("rung", num, den, "transferred", seen[-1], "nnz'", cl3.numel())
    assert seen[0] == 0 and seen == sorted(seen) and seen[-1] > seen[1]


@pytest.mark.parametrize("name,mult", [("c4", 1), ("c4", 10), ("c3", 5)])
def test_full_size(gt, name, mult):
    # the workload reordered on the GPU, then rewritten at mult x beta_G with k = 8, d_b = 16
    w = make_workload(name)
    g = w.graph
    say("full size", name, g.n, g.nnz, "x", mult)
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2 = gt.permute_csr(rp, cl, perm, iperm)
    r, c = rp2.cpu().numpy(), cl2.cpu().numpy()
    _, cl3, info = check(gt, r, c, 8, 16, mult * g.nnz, g.n * g.n, progress=lambda m: say("  oracle:", m))
    say("  transferred", int(info["transfer"].sum()), "nnz'", cl3.numel())
    assert info["transfer"].any()


def test_attention_on_the_rewritten_graph(gt):
    # the exact attention path on E' (the oracle's attention over E', §3.4's modified edge set)
    w = make_workload("c2", 0.05)
    g = w.graph
    q, k, v, do = w.tensors()
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2 = gt.permute_csr(rp, cl, perm, iperm)
    r, c = rp2.cpu().numpy(), cl2.cpu().numpy()
    rp3, cl3, info = check(gt, r, c, 8, 16, 5 * g.nnz, g.n * g.n)
    assert info["transfer"].any()
    pr = perm.cpu().numpy()
    qp, kp, vp, dop = (x[pr] for x in (q, k, v, do))
    scale = 1.0 / np.sqrt(w.dim)
    plan = gt.build_tiles(rp3, cl3, 128, 10_000)
    Q, K, V, dO = (dev_feat(x, w.dtype) for x in (qp, kp, vp, dop))
    O, L = gt.sparse_attn_fwd(plan, Q, K, V, scale)
    grads = gt.sparse_attn_bwd(plan, Q, K, V, dO, L, scale)
    torch.cuda.synchronize()
    r3, c3 = rp3.cpu().numpy(), cl3.cpu().numpy()
    O_ref, L_ref = OA.sparse_attn_fwd(r3, c3, qp, kp, vp, scale)
    ref = OA.sparse_attn_bwd(r3, c3, qp, kp, vp, dop, scale)
    assert_close(host(O), O_ref, w.dtype, "O")
    assert_close(L.cpu().numpy(), L_ref, w.dtype, "LSE")
    for name, x, rr in zip(("dQ", "dK", "dV"), grads, ref):
        assert_close(host(x), rr, w.dtype, name)
