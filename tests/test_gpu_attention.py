"""GPU neighbourhood softmax attention (§3.2) vs the fp64 oracle, forward and
backward, across tile plans (§3.4: every density threshold gives the same
result), dtypes, head counts and widths, plus edge cases: empty rows, rows and
columns longer than one wavefront slice can take, ragged sizes, a single node.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import plan as OP
from oracle import reorder as OR
from synth import csr_from_pairs, make_workload
from synth.tensors import normal_tensor
from tests.helpers import assert_close, dev_csr, dev_feat, host

pytestmark = pytest.mark.gpu

CSR_ONLY = 1_000_001  # threshold above 100%: no dense tile, every edge on the edge kernels
SWEEP = (0, 10_000, 50_000, CSR_ONLY)  # every non-empty tile dense, 1%, 5%, none


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def feats(n, H, d, dtype, seed):
    return [normal_tensor((n, H, d), (seed, t), dtype) for t in range(4)]


def run_case(gt, rowptr, col, H, d, dtype, taus=(CSR_ONLY,), T=128, seed=0, bwd=True):
    n = len(rowptr) - 1
    q, k, v, do = feats(n, H, d, dtype, seed)
    scale = 1.0 / np.sqrt(d)
    O_ref, L_ref = OA.sparse_attn_fwd(rowptr, col, q, k, v, scale)
    grads_ref = OA.sparse_attn_bwd(rowptr, col, q, k, v, do, scale) if bwd else None
    rp, cl = dev_csr(rowptr, col)
    Q, K, V, dO = (dev_feat(x, dtype) for x in (q, k, v, do))
    for tau in taus:
        say("case", n, len(col), H, d, dtype, T, tau)
        plan = gt.build_tiles(rp, cl, T, tau)
        O, L = gt.sparse_attn_fwd(plan, Q, K, V, scale)
        torch.cuda.synchronize()
        assert_close(host(O), O_ref, dtype, f"O tau={tau}")
        assert_close(L.cpu().numpy(), L_ref, dtype, f"LSE tau={tau}")
        if bwd:
            dQ, dK, dV = gt.sparse_attn_bwd(plan, Q, K, V, dO, L, scale)
            torch.cuda.synchronize()
            for name, x, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), grads_ref):
                assert_close(host(x), r, dtype, f"{name} tau={tau}")
            # the two halves as the benchmark calls them (the row pass's statistic handed to the column pass):
            # D against the oracle's <dO_i, O_i>, the gradients equal to the combined call's bit for bit
            dQ2, Dst = gt.sparse_attn_bwd_rows(plan, Q, K, V, dO, L, scale)
            dK2, dV2 = gt.sparse_attn_bwd_cols(plan, Q, K, V, dO, L, Dst, scale)
            torch.cuda.synchronize()
            assert_close(Dst.cpu().numpy(), np.einsum("nhc,nhc->nh", np.asarray(do, np.float64), O_ref), dtype,
                         f"D tau={tau}")
            for name, a, b in zip(("dQ", "dK", "dV"), (dQ, dK, dV), (dQ2, dK2, dV2)):
                assert torch.equal(a, b), f"{name} of the split backward differs from the combined call, tau={tau}"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H,d", [(1, 64), (2, 32), (4, 32), (8, 32), (8, 64), (16, 32), (16, 64), (1, 32)])
def test_small_graph_all_shapes(gt, dtype, H, d):
    g = make_workload("c1", 0.1).graph
    run_case(gt, g.rowptr, g.col, H, d, dtype, taus=SWEEP, seed=H * 100 + d)


@pytest.mark.parametrize("T", [64, 128])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tile_sizes_on_clustered_graph(gt, T, dtype):
    # a block-model graph in planted order: diagonal tiles well above 5%
    w = make_workload("c5", 0.03)
    g = w.graph
    order = np.lexsort((np.arange(g.n), g.block))
    inv = np.empty(g.n, np.int64)
    inv[order] = np.arange(g.n)
    rp, cl = OP.permute_csr(g.rowptr, g.col, order, inv)
    run_case(gt, rp, cl, 4, 64, dtype, taus=SWEEP, T=T, seed=T)


def test_c1_full_fp32_forward(gt):
    w = make_workload("c1")
    q, k, v, _ = w.tensors()
    g = w.graph
    O_ref, L_ref = OA.sparse_attn_fwd(g.rowptr, g.col, q, k, v, 1 / 8)
    rp, cl = dev_csr(g.rowptr, g.col)
    plan = gt.build_tiles(rp, cl, 128, CSR_ONLY)
    O, L = gt.sparse_attn_fwd(plan, dev_feat(q, "f32"), dev_feat(k, "f32"), dev_feat(v, "f32"), 1 / 8)
    assert_close(host(O), O_ref, "f32", "O")
    assert_close(L.cpu().numpy(), L_ref, "f32", "LSE")


@pytest.mark.parametrize("name,scale", [("c2", 0.02), ("c3", 0.01), ("c4", 0.005), ("c5", 0.05)])
def test_workload_shapes_bf16(gt, name, scale):
    w = make_workload(name, scale)
    run_case(gt, w.graph.rowptr, w.graph.col, w.heads, w.dim, w.dtype, taus=(10_000, CSR_ONLY), seed=w.seed)


def test_empty_rows_single_node_and_ragged(gt):
    # rows 3 and 77 are empty; n = 131 is not a multiple of any tile or wave size
    u = np.array([0, 1, 2, 5, 5, 9, 100, 130, 130])
    v = np.array([1, 2, 4, 6, 7, 9, 101, 0, 129])
    rowptr, col = csr_from_pairs(131, u, v, symmetric=False, self_loops=False)
    for dtype in ("f32", "bf16"):
        for T in (64, 128):
            run_case(gt, rowptr, col, 4, 32, dtype, taus=SWEEP, T=T, seed=3)
    rowptr, col = csr_from_pairs(1, [], [])
    run_case(gt, rowptr, col, 8, 64, "bf16", taus=SWEEP, seed=4)


def test_long_rows_and_columns(gt):
    # hub 0 attends to 3000 nodes and is attended by them; node 5 has 300 in-edges only
    n = 4000
    u = np.concatenate([np.zeros(3000, np.int64), np.arange(1000, 1300)])
    v = np.concatenate([np.arange(1, 3001), np.full(300, 5)])
    rowptr, col = csr_from_pairs(n, u[:3000], v[:3000], symmetric=True, self_loops=True)
    r2, c2 = csr_from_pairs(n, u[3000:], v[3000:], symmetric=False, self_loops=False)
    dense = np.zeros((n, n), bool)
    for rp_, cl_ in ((rowptr, col), (r2, c2)):
        rows = np.repeat(np.arange(n), np.diff(rp_))
        dense[rows, cl_] = True
    uu, vv = np.nonzero(dense)
    rowptr, col = csr_from_pairs(n, uu, vv, symmetric=False, self_loops=False)
    for dtype, H, d in (("f32", 2, 64), ("bf16", 8, 32), ("bf16", 16, 64)):
        run_case(gt, rowptr, col, H, d, dtype, taus=(0, 5000, CSR_ONLY), seed=H + d)


def test_hub_tile_rows_and_columns_in_chunks(gt):
    # 96 hub rows attend to half of all nodes and 64 hub columns are attended by half of all rows, over a sparse
    # background; n = 2117 is ragged for both tile sizes.  Each hub tile row (column) holds ~17-34 dense tiles,
    # so its dense tiles are dealt out to several workgroups whose partial states are merged.
    n = 2117
    rng = np.random.default_rng(5)
    hub_r = np.repeat(np.arange(96), n // 2)
    hub_rc = rng.integers(0, n, size=len(hub_r))
    hub_c = np.repeat(np.arange(200, 264), n // 2)
    hub_cr = rng.integers(0, n, size=len(hub_c))
    bu, bv = rng.integers(0, n, size=6 * n), rng.integers(0, n, size=6 * n)
    u = np.concatenate([hub_r, hub_cr, bu])
    v = np.concatenate([hub_rc, hub_c, bv])
    rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=True)
    for T in (64, 128):
        run_case(gt, rowptr, col, 4, 64, "bf16", taus=(0, 50_000), T=T, seed=T + 1)
    run_case(gt, rowptr, col, 8, 32, "bf16", taus=(10_000,), T=128, seed=9)
    # every merge geometry: D / 4 lanes per row, T / (256 / (D / 4)) row blocks per (tile row, head)
    for H, d, T in ((16, 64, 64), (1, 32, 64), (2, 64, 128), (16, 32, 128)):
        run_case(gt, rowptr, col, H, d, "bf16", taus=(0,), T=T, seed=H * d + T, bwd=True)


def test_bitwise_deterministic(gt):
    w = make_workload("c4", 0.01)
    g = w.graph
    q, k, v, do = w.tensors()
    rp, cl = dev_csr(g.rowptr, g.col)
    plan = gt.build_tiles(rp, cl, 128, 10_000)
    assert plan.n_dense > 0
    Q, K, V, dO = (dev_feat(x, "bf16") for x in (q, k, v, do))
    outs = []
    for _ in range(2):
        O, L = gt.sparse_attn_fwd(plan, Q, K, V)
        outs.append((O, L, *gt.sparse_attn_bwd(plan, Q, K, V, dO, L)))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_pipeline_reorder_then_attention_is_equivariant(gt):
    # reorder + relabel + gather on the GPU, attention in the new order, scatter back:
    # equals the oracle on the original order.
    w = make_workload("c5", 0.05)
    g = w.graph
    q, k, v, do = w.tensors()
    scale = 1 / 8
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2 = gt.permute_csr(rp, cl, perm, iperm)
    plan = gt.build_tiles(rp2, cl2, 128, 10_000)
    assert plan.n_dense > 0
    Q, K, V, dO = (gt.gather_rows(dev_feat(x, "bf16"), perm) for x in (q, k, v, do))
    O, L = gt.sparse_attn_fwd(plan, Q, K, V, scale)
    dQ, dK, dV = gt.sparse_attn_bwd(plan, Q, K, V, dO, L, scale)
    O_ref, L_ref = OA.sparse_attn_fwd(g.rowptr, g.col, q, k, v, scale)
    ref = OA.sparse_attn_bwd(g.rowptr, g.col, q, k, v, do, scale)
    assert_close(host(gt.scatter_rows(O, perm)), O_ref, "bf16", "O")
    assert_close(gt.scatter_rows(L, perm).cpu().numpy(), L_ref, "bf16", "LSE")
    for name, x, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref):
        assert_close(host(gt.scatter_rows(x, perm)), r, "bf16", name)


@pytest.mark.parametrize("name,tau", [("c2", 10_000), ("c3", 10_000), ("c4", 50_000), ("c4", 10_000),
                                      ("c5", 10_000), ("b1", 10_000), ("b2", 50_000)])
def test_full_size_workloads_sampled(gt, name, tau):
    # The workloads at their full sizes through the library's whole pipeline, in the launch configuration the
    # benchmark times (reorder, relabel, 128-wide tiles at the workload's threshold, row gather, the forward,
    # then the backward's row and column calls), with the outputs scattered back to the input order.  The oracle computes 192
    # random rows (forward, dQ) and columns (dK, dV) one by one on the original graph, plus the eight rows of
    # largest degree (hubs on the power-law graph, the global token of the batched graphs).  A column attended
    # by more than 65,536 rows (the global token's) is left to the small batched test, which checks it in
    # full: its dK and dV need the softmax statistics of every row.
    w = make_workload(name)
    g = w.graph
    q, k, v, do = w.tensors()
    scale = 1.0 / np.sqrt(w.dim)
    say("full size", name, g.n, g.nnz, tau)
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2 = gt.permute_csr(rp, cl, perm, iperm)
    plan = gt.build_tiles(rp2, cl2, 128, tau)
    Q, K, V, dO = (gt.gather_rows(dev_feat(x, w.dtype), perm) for x in (q, k, v, do))
    O, L = gt.sparse_attn_fwd(plan, Q, K, V, scale)
    dQ, Dst = gt.sparse_attn_bwd_rows(plan, Q, K, V, dO, L, scale)
    dK, dV = gt.sparse_attn_bwd_cols(plan, Q, K, V, dO, L, Dst, scale)
    outs = [gt.scatter_rows(x, perm) for x in (O, L, dQ, dK, dV)]
    torch.cuda.synchronize()
    say("  dense tiles", plan.n_dense, "long rows", plan.c.n_long_rows, "long cols", plan.c.n_long_cols)
    rng = np.random.default_rng(11)
    deg = np.diff(g.rowptr)
    rows = np.unique(np.concatenate([rng.choice(g.n, size=192, replace=False), np.argsort(deg)[-8:]]))
    cols = rows[deg[rows] <= 65_536]
    say("  oracle on", len(rows), "rows and", len(cols), "columns")
    O_ref, L_ref = OA.sparse_attn_fwd(g.rowptr, g.col, q, k, v, scale, rows=rows)
    dq_ref, dk_ref, dv_ref = OA.sparse_attn_bwd_sampled(g.rowptr, g.col, q, k, v, do, scale, rows, cols)
    say("  oracle done")
    idx = torch.from_numpy(rows).cuda()
    cdx = torch.from_numpy(cols).cuda()
    for nm, x, r in zip(("O", "dQ"), (outs[0], outs[2]), (O_ref, dq_ref)):
        assert_close(host(x[idx]), r, w.dtype, f"{name} {nm}")
    for nm, x, r in zip(("dK", "dV"), (outs[3], outs[4]), (dk_ref, dv_ref)):
        assert_close(host(x[cdx]), r, w.dtype, f"{name} {nm}")
    assert_close(outs[1][idx].cpu().numpy(), L_ref, w.dtype, f"{name} LSE")


def test_batched_small_graphs_with_global_token(gt):
    # Graph-level batching: 400 molecule-sized graphs as one block-diagonal graph plus a global token whose
    # row and column hold every node (a 9,809-edge row and column, cut into chunks), every tile plan.
    w = make_workload("b1", 0.01)
    g = w.graph
    run_case(gt, g.rowptr, g.col, 8, 32, "bf16", taus=SWEEP, seed=21)
    run_case(gt, g.rowptr, g.col, 2, 64, "f32", taus=(10_000, CSR_ONLY), seed=22)


def test_gather_probe_runs_on_every_shape(gt):
    # measurement-only entry point: must run (in bounds) for every supported shape and leave the features alone
    g = make_workload("c1", 0.1).graph
    rp, cl = dev_csr(g.rowptr, g.col)
    plan = gt.build_tiles(rp, cl, 128, CSR_ONLY)
    for dtype in ("f32", "bf16"):
        for H, d in ((1, 32), (8, 32), (16, 64)):
            a, b = (dev_feat(x, dtype) for x in feats(g.n, H, d, dtype, 7)[:2])
            a0, b0 = a.clone(), b.clone()
            gt.gather_probe(plan, a, b)
            torch.cuda.synchronize()
            assert torch.equal(a, a0) and torch.equal(b, b0)
