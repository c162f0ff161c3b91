"""GPU attention with a per-edge additive bias (the graph encoding added to
the scaled product, §2.1 Eq. (3), kept in the attention's sparse layout, §3.3)
vs the fp64 oracle: forward, the three feature gradients and dB, on small
graphs, long rows and columns, the relabelling pipeline that carries the bias
with its edges, and the workloads at full size on sampled rows and columns.
"""

import sys

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import plan as OP
from synth import csr_from_pairs, make_workload
from synth.tensors import normal_tensor
from tests.helpers import assert_close, dev_csr, dev_feat, grad_term_rms, host

pytestmark = pytest.mark.gpu

CSR_ONLY = 1_000_001  # no dense tile: every edge on the edge kernels
SWEEP = (0, 10_000, 50_000, CSR_ONLY)  # every non-empty tile dense, 1%, 5%, none


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev_bias(b):
    return torch.from_numpy(np.ascontiguousarray(b, dtype=np.float32)).cuda()


def run_bias_case(gt, rowptr, col, H, d, dtype, seed, bias_sigma=1.0, taus=(CSR_ONLY,), T=128):
    # The bias is one array in the input CSR's edge order whatever the plan: the dense tiles (sp_pos and
    # tile_pos in the plan) and the remainder take their edges' values from it, and dB comes back in it.
    n = len(rowptr) - 1
    q, k, v, do = (normal_tensor((n, H, d), (seed, t), dtype) for t in range(4))
    b = bias_sigma * normal_tensor((len(col), H), (seed, 4), "f32")
    scale = 1.0 / np.sqrt(d)
    O_ref, L_ref = OA.sparse_attn_fwd(rowptr, col, q, k, v, scale, bias=b)
    ref = OA.sparse_attn_bwd(rowptr, col, q, k, v, do, scale, bias=b)
    floors = grad_term_rms(rowptr, col, q, k, v, do, scale)
    rp, cl = dev_csr(rowptr, col)
    Q, K, V, dO = (dev_feat(x, dtype) for x in (q, k, v, do))
    B = dev_bias(b)
    for tau in taus:
        say("bias case", n, len(col), H, d, dtype, T, tau)
        plan = gt.build_tiles(rp, cl, T, tau, edge_positions=True)
        if tau == CSR_ONLY:
            assert plan.n_dense == 0 and plan.nnz_sparse == len(col)
        csc = gt.edge_map(plan)
        O, L = gt.sparse_attn_fwd_bias(plan, Q, K, V, B, scale)
        grads = gt.sparse_attn_bwd_bias(plan, csc, Q, K, V, B, dO, L, scale)
        torch.cuda.synchronize()
        assert_close(host(O), O_ref, dtype, f"O tau={tau}")
        assert_close(L.cpu().numpy(), L_ref, dtype, f"LSE tau={tau}")
        for name, x, r, rho in zip(("dQ", "dK", "dV", "dB"), grads, ref, floors):
            assert_close(host(x), r, dtype, f"{name} tau={tau}", rho=rho)


def test_edge_map_is_the_stable_column_order(gt):
    g = make_workload("c3", 0.02).graph
    rp, cl = dev_csr(g.rowptr, g.col)
    for tau in (10_000, CSR_ONLY):
        plan = gt.build_tiles(rp, cl, 128, tau)
        csc = gt.edge_map(plan).cpu().numpy()
        sp_col = plan.arrays["sp_col"].cpu().numpy()
        sp_rowptr = plan.arrays["sp_rowptr"].cpu().numpy()
        # the CSC order of the remainder: by column, rows ascending (CSR positions ascending) in each column
        assert np.array_equal(csc, np.argsort(sp_col, kind="stable"))
        rows = np.repeat(np.arange(g.n), np.diff(sp_rowptr))
        assert np.array_equal(rows[csc], plan.arrays["sp_row"].cpu().numpy())


def test_permute_edges_carries_positions(gt):
    g = make_workload("c5", 0.03).graph
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2, src = gt.permute_csr_edges(rp, cl, perm, iperm)
    rpa, cla = gt.permute_csr(rp, cl, perm, iperm)
    assert torch.equal(rp2, rpa) and torch.equal(cl2, cla)
    src, rp2, cl2 = src.cpu().numpy(), rp2.cpu().numpy(), cl2.cpu().numpy()
    perm_h, iperm_h = perm.cpu().numpy(), iperm.cpu().numpy()
    assert np.array_equal(np.sort(src), np.arange(g.nnz))
    new_row = np.repeat(np.arange(g.n), np.diff(rp2))
    old_row = np.repeat(np.arange(g.n), np.diff(g.rowptr))
    # every new edge (r, c) came from old edge (perm[r], perm[c]) (columns are unique within a row)
    assert np.array_equal(old_row[src], perm_h[new_row])
    assert np.array_equal(iperm_h[g.col[src]], cl2)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H,d", [(1, 64), (4, 32), (8, 32), (8, 64), (16, 32)])
def test_bias_small_graph(gt, dtype, H, d):
    g = make_workload("c1", 0.1).graph
    run_bias_case(gt, g.rowptr, g.col, H, d, dtype, seed=300 + H * 10 + d, taus=SWEEP)


@pytest.mark.parametrize("T", [64, 128])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bias_on_dense_tiles_of_a_clustered_graph(gt, T, dtype):
    # a block-model graph in planted order: diagonal tiles above 5%, so the bias reaches the matrix-core tiles
    w = make_workload("c5", 0.03)
    g = w.graph
    order = np.lexsort((np.arange(g.n), g.block))
    inv = np.empty(g.n, np.int64)
    inv[order] = np.arange(g.n)
    rp, cl = OP.permute_csr(g.rowptr, g.col, order, inv)
    run_bias_case(gt, rp, cl, 4, 64, dtype, seed=T + 7, taus=SWEEP, T=T)


def test_bias_on_hub_tiles_in_chunks(gt):
    # hub tile rows and columns (several dense tiles per tile row and column, dealt to several workgroups and
    # merged) with a bias of spread 4
    n = 2117
    rng = np.random.default_rng(15)
    hub_r = np.repeat(np.arange(96), n // 2)
    hub_rc = rng.integers(0, n, size=len(hub_r))
    hub_c = np.repeat(np.arange(200, 264), n // 2)
    hub_cr = rng.integers(0, n, size=len(hub_c))
    bu, bv = rng.integers(0, n, size=6 * n), rng.integers(0, n, size=6 * n)
    u = np.concatenate([hub_r, hub_cr, bu])
    v = np.concatenate([hub_rc, hub_c, bv])
    rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=True)
    run_bias_case(gt, rowptr, col, 8, 32, "bf16", seed=61, bias_sigma=4.0, taus=(0, 50_000), T=128)
    run_bias_case(gt, rowptr, col, 2, 64, "f32", seed=62, taus=(0, 50_000), T=64)


def test_plan_edge_positions(gt):
    # sp_pos and tile_pos of a plan with dense tiles and long rows, against positions found on the host
    g = make_workload("b1", 0.01).graph
    assert np.diff(g.rowptr).max() > 2048  # the global token's row takes the plan's long-row fill
    rp, cl = dev_csr(g.rowptr, g.col)
    for T, tau in ((128, 10_000), (64, 50_000), (128, 0)):
        plan = gt.build_tiles(rp, cl, T, tau, edge_positions=True)
        assert plan.n_dense > 0
        arr = plan.to_numpy()
        rows = np.repeat(np.arange(g.n), np.diff(g.rowptr))
        dense = set(zip(np.repeat(np.arange(len(arr["tile_rowptr"]) - 1), np.diff(arr["tile_rowptr"])).tolist(),
                        arr["tile_col"].tolist()))
        in_tile = np.array([(int(r) // T, int(c) // T) in dense for r, c in zip(rows, g.col)])
        np.testing.assert_array_equal(arr["sp_pos"], np.flatnonzero(~in_tile))
        tile_index = {t: k for k, t in enumerate(zip(np.repeat(np.arange(len(arr["tile_rowptr"]) - 1),
                                                               np.diff(arr["tile_rowptr"])).tolist(),
                                                     arr["tile_col"].tolist()))}
        want = np.zeros(plan.n_dense * T, np.int64)
        for e in np.flatnonzero(in_tile)[::-1]:  # the smallest position of each (tile, row) wins
            r, c = int(rows[e]), int(g.col[e])
            want[tile_index[(r // T, c // T)] * T + r % T] = e
        np.testing.assert_array_equal(arr["tile_pos"], want)
        csc = gt.edge_map(plan).cpu().numpy()
        rem = np.argsort(arr["sp_col"], kind="stable")
        np.testing.assert_array_equal(csc, arr["sp_pos"][rem])


def test_bias_ragged_empty_rows_single_node(gt):
    u = np.array([0, 1, 2, 5, 5, 9, 100, 130, 130])
    v = np.array([1, 2, 4, 6, 7, 9, 101, 0, 129])
    rowptr, col = csr_from_pairs(131, u, v, symmetric=False, self_loops=False)
    run_bias_case(gt, rowptr, col, 4, 32, "f32", seed=31)
    run_bias_case(gt, rowptr, col, 2, 64, "bf16", seed=32)
    rowptr, col = csr_from_pairs(1, [], [])
    run_bias_case(gt, rowptr, col, 8, 64, "bf16", seed=33)


def test_bias_long_rows_and_columns(gt):
    # hub 0 attends to (and is attended by) 3,000 nodes: chunked rows and columns carry the bias too
    n = 4000
    rowptr, col = csr_from_pairs(n, np.zeros(3000, np.int64), np.arange(1, 3001), symmetric=True,
                                 self_loops=True)
    for dtype, H, d in (("f32", 2, 64), ("bf16", 8, 32)):
        run_bias_case(gt, rowptr, col, H, d, dtype, seed=40 + H)


def test_large_bias_moves_the_max(gt):
    # bias of spread 8 (about 11.5 in the exp2 domain) makes the lazy running max move within rows
    g = make_workload("c1", 0.1).graph
    run_bias_case(gt, g.rowptr, g.col, 4, 32, "f32", seed=51, bias_sigma=8.0)


def test_zero_bias_matches_plain_path(gt):
    # A zero bias: the forward is bitwise the plain path's; the backward may differ by the rounding of the
    # score (the bias path's product and sum can be fused), so it is checked at the bf16 tolerance, and dB
    # against the oracle's dS.
    w = make_workload("c4", 0.01)
    g = w.graph
    q, k, v, do = w.tensors()
    rp, cl = dev_csr(g.rowptr, g.col)
    plan = gt.build_tiles(rp, cl, 128, CSR_ONLY)
    Q, K, V, dO = (dev_feat(x, "bf16") for x in (q, k, v, do))
    B = torch.zeros((plan.nnz_sparse, w.heads), dtype=torch.float32, device="cuda")
    O, L = gt.sparse_attn_fwd(plan, Q, K, V)
    Ob, Lb = gt.sparse_attn_fwd_bias(plan, Q, K, V, B)
    assert torch.equal(O, Ob) and torch.equal(L, Lb)
    plain = gt.sparse_attn_bwd(plan, Q, K, V, dO, L)
    withb = gt.sparse_attn_bwd_bias(plan, gt.edge_map(plan), Q, K, V, B, dO, L)
    for name, a, b in zip(("dQ", "dK", "dV"), plain, withb[:3]):
        assert_close(host(b), host(a), "bf16", name)
    ref = OA.sparse_attn_bwd(g.rowptr, g.col, q, k, v, do, 1 / np.sqrt(w.dim), bias=np.zeros((g.nnz, w.heads)))
    assert_close(host(withb[3]), ref[3], "bf16", "dB")


def test_bias_needs_edge_positions_on_a_plan_with_dense_tiles(gt):
    w = make_workload("c4", 0.01)
    g = w.graph
    rp, cl = dev_csr(g.rowptr, g.col)
    plan = gt.build_tiles(rp, cl, 128, 10_000)
    assert plan.n_dense > 0
    q, k, v, _ = w.tensors()
    Q, K, V = (dev_feat(x, "bf16") for x in (q, k, v))
    B = torch.zeros((g.nnz, w.heads), dtype=torch.float32, device="cuda")
    with pytest.raises(gt.GtError) as e:
        gt.sparse_attn_fwd_bias(plan, Q, K, V, B)
    assert e.value.status == gt.GT_ERR_INVALID_ARG


def test_bias_pipeline_relabel_carries_the_bias(gt):
    # reorder + relabel (with the edge map) on the GPU, the bias gathered into the new edge order, attention on
    # a plan with dense tiles, everything scattered back: equals the oracle on the original graph and bias order.
    w = make_workload("c5", 0.05)
    g = w.graph
    q, k, v, do = w.tensors()
    b = w.edge_bias()
    scale = 1 / 8
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2, src = gt.permute_csr_edges(rp, cl, perm, iperm)
    plan = gt.build_tiles(rp2, cl2, 128, 10_000, edge_positions=True)
    assert plan.n_dense > 0
    Q, K, V, dO = (gt.gather_rows(dev_feat(x, "bf16"), perm) for x in (q, k, v, do))
    B = gt.gather_rows(dev_bias(b), src)
    O, L = gt.sparse_attn_fwd_bias(plan, Q, K, V, B, scale)
    dQ, dK, dV, dB = gt.sparse_attn_bwd_bias(plan, gt.edge_map(plan), Q, K, V, B, dO, L, scale)
    O_ref, L_ref = OA.sparse_attn_fwd(g.rowptr, g.col, q, k, v, scale, bias=b)
    ref = OA.sparse_attn_bwd(g.rowptr, g.col, q, k, v, do, scale, bias=b)
    assert_close(host(gt.scatter_rows(O, perm)), O_ref, "bf16", "O")
    assert_close(gt.scatter_rows(L, perm).cpu().numpy(), L_ref, "bf16", "LSE")
    for name, x, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref[:3]):
        assert_close(host(gt.scatter_rows(x, perm)), r, "bf16", name)
    assert_close(host(gt.scatter_rows(dB, src)), ref[3], "bf16", "dB")


@pytest.mark.parametrize("name", ["c3", "b1"])
def test_bias_full_size_sampled(gt, name):
    # Full-size workloads with a bias through the whole pipeline (reorder, relabel with the edge map, bias
    # gather, all-remainder plan, forward, backward, scatter back); the oracle computes sampled rows (O, LSE,
    # dQ and dB of their edges) and columns (dK, dV), plus the eight rows of largest degree.
    w = make_workload(name)
    g = w.graph
    q, k, v, do = w.tensors()
    b = w.edge_bias()
    scale = 1.0 / np.sqrt(w.dim)
    say("full size with bias", name, g.n, g.nnz)
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, _ = gt.reorder(rp, cl)
    rp2, cl2, src = gt.permute_csr_edges(rp, cl, perm, iperm)
    plan = gt.build_tiles(rp2, cl2, 128, CSR_ONLY)
    Q, K, V, dO = (gt.gather_rows(dev_feat(x, w.dtype), perm) for x in (q, k, v, do))
    B = gt.gather_rows(dev_bias(b), src)
    O, L = gt.sparse_attn_fwd_bias(plan, Q, K, V, B, scale)
    dQ, dK, dV, dB = gt.sparse_attn_bwd_bias(plan, gt.edge_map(plan), Q, K, V, B, dO, L, scale)
    outs = [gt.scatter_rows(x, perm) for x in (O, L, dQ, dK, dV)]
    dB = gt.scatter_rows(dB, src)
    torch.cuda.synchronize()
    say("  long rows", plan.c.n_long_rows, "long cols", plan.c.n_long_cols)
    rng = np.random.default_rng(12)
    deg = np.diff(g.rowptr)
    rows = np.unique(np.concatenate([rng.choice(g.n, size=192, replace=False), np.argsort(deg)[-8:]]))
    cols = rows[deg[rows] <= 65_536]
    say("  oracle on", len(rows), "rows and", len(cols), "columns")
    O_ref, L_ref = OA.sparse_attn_fwd(g.rowptr, g.col, q, k, v, scale, rows=rows, bias=b)
    dq_ref, dk_ref, dv_ref, (epos, db_ref) = OA.sparse_attn_bwd_sampled(g.rowptr, g.col, q, k, v, do, scale, rows,
                                                                        cols, bias=b)
    say("  oracle done")
    idx = torch.from_numpy(rows).cuda()
    cdx = torch.from_numpy(cols).cuda()
    for nm, x, r in zip(("O", "dQ"), (outs[0], outs[2]), (O_ref, dq_ref)):
        assert_close(host(x[idx]), r, w.dtype, f"{name} {nm}")
    for nm, x, r in zip(("dK", "dV"), (outs[3], outs[4]), (dk_ref, dv_ref)):
        assert_close(host(x[cdx]), r, w.dtype, f"{name} {nm}")
    assert_close(outs[1][idx].cpu().numpy(), L_ref, w.dtype, f"{name} LSE")
    assert_close(host(dB[torch.from_numpy(epos).cuda()]), db_ref, w.dtype, f"{name} dB")
