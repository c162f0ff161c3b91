"""Pins of the relabelling and tile-plan oracle (§3.3 layout reorganisation,
§3.4 cluster sparsity and transfer threshold) against independent
constructions: scipy's sparse permutation and transpose, brute-force tile counts
from the dense adjacency, and the threshold's boundary cases."""

import numpy as np
import pytest
import scipy.sparse as sp

from oracle import plan as P
from synth import csr_from_pairs, make_workload


def rand_csr(n, p, seed, symmetric=False):
    rng = np.random.default_rng(seed)
    m = rng.random((n, n)) < p
    u, v = np.nonzero(m)
    return csr_from_pairs(n, u, v, symmetric=symmetric, self_loops=True)


def dense_of(rowptr, col, n):
    return sp.csr_matrix((np.ones(len(col)), np.asarray(col), np.asarray(rowptr)), shape=(n, n)).toarray() > 0


def test_permute_csr_is_p_a_pt():
    n = 57
    rowptr, col = rand_csr(n, 0.1, 1)
    perm = np.random.default_rng(2).permutation(n)
    iperm = np.empty(n, np.int64)
    iperm[perm] = np.arange(n)
    rp, c = P.permute_csr(rowptr, col, perm, iperm)
    A = sp.csr_matrix((np.ones(len(col)), col, rowptr), shape=(n, n))
    Pm = sp.csr_matrix((np.ones(n), perm, np.arange(n + 1)), shape=(n, n))  # row r picks old row perm[r]
    ref = (Pm @ A @ Pm.T).tocsr()
    ref.sort_indices()
    np.testing.assert_array_equal(rp, ref.indptr)
    np.testing.assert_array_equal(c, ref.indices)


@pytest.mark.parametrize("n,T,tau_ppm,seed", [(300, 64, 20000, 0), (511, 128, 5000, 1), (200, 64, 0, 2),
                                             (129, 128, 10000, 3), (64, 64, 1_000_001, 4)])
def test_tiles_against_brute_force(n, T, tau_ppm, seed):
    rowptr, col = rand_csr(n, 0.03, seed)
    # plant a denser block so that some tiles cross the threshold
    dense = dense_of(rowptr, col, n)
    dense[:40, :40] |= np.random.default_rng(seed).random((40, 40)) < 0.4
    u, v = np.nonzero(dense)
    rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    plan = P.build_tiles(rowptr, col, T, tau_ppm)
    R = (n + T - 1) // T
    pad = np.zeros((R * T, R * T), dtype=bool)
    pad[:n, :n] = dense
    blocks = pad.reshape(R, T, R, T).transpose(0, 2, 1, 3)
    want = []
    for I in range(R):
        for J in range(R):
            cnt = int(blocks[I, J].sum())
            area = min(T, n - I * T) * min(T, n - J * T)
            if cnt >= 1 and cnt * 10**6 >= tau_ppm * area:
                want.append((I, J, cnt))
    got_I = np.repeat(np.arange(R), np.diff(plan["tile_rowptr"]))
    assert list(zip(got_I.tolist(), plan["tile_col"].tolist(), plan["tile_nnz"].tolist())) == want
    # masks reproduce each tile's block; the remainder is everything else
    words = T // 32
    masks = plan["tile_mask"].reshape(-1, T, words)
    rebuilt = np.zeros_like(pad)
    for k, (I, J, _) in enumerate(want):
        bits = ((masks[k][:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(T, T).astype(bool)
        assert bits.sum() == plan["tile_nnz"][k]
        rebuilt[I * T:(I + 1) * T, J * T:(J + 1) * T] |= bits
    rem = dense_of(plan["sp_rowptr"], plan["sp_col"], n)
    assert not (rem & rebuilt[:n, :n]).any()
    np.testing.assert_array_equal(rem | rebuilt[:n, :n], dense)
    assert not rebuilt[n:, :].any() and not rebuilt[:, n:].any()
    assert plan["tile_nnz"].sum() + len(plan["sp_col"]) == len(col)
    # transpose of the remainder (scipy) and the column-grouped tile list
    csc = sp.csr_matrix((np.ones(len(plan["sp_col"])), plan["sp_col"], plan["sp_rowptr"]), shape=(n, n)).tocsc()
    csc.sort_indices()
    np.testing.assert_array_equal(plan["sp_colptr"], csc.indptr)
    np.testing.assert_array_equal(plan["sp_row"], csc.indices)
    order = sorted(range(len(want)), key=lambda k: (want[k][1], want[k][0]))
    assert plan["tileT_idx"].tolist() == order
    np.testing.assert_array_equal(plan["tileT_ptr"], np.concatenate([[0], np.cumsum(np.bincount(
        [w[1] for w in want], minlength=R))]))


def test_threshold_boundary_is_inclusive():
    # one 64x64 tile with exactly 41 edges: density 41/4096 = 10009.765... ppm
    n, T = 64, 64
    u = np.arange(41) % 64
    v = (np.arange(41) * 7) % 64
    rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    cnt = len(col)
    # the largest tau_ppm that keeps the tile dense: cnt*1e6 >= tau*4096
    tau_edge = (cnt * 10**6) // (T * T)
    assert len(P.build_tiles(rowptr, col, T, tau_edge)["tile_col"]) == 1
    assert len(P.build_tiles(rowptr, col, T, tau_edge + 1)["tile_col"]) == 0
    # exact equality: 4096 edges at tau = 1e6 (fully dense) and 2048 at tau = 500000
    full = np.ones((64, 64), bool)
    u, v = np.nonzero(full)
    rp, c = csr_from_pairs(64, u, v, symmetric=False, self_loops=False)
    assert len(P.build_tiles(rp, c, 64, 1_000_000)["tile_col"]) == 1
    half = np.zeros((64, 64), bool)
    half[:, :32] = True
    u, v = np.nonzero(half)
    rp, c = csr_from_pairs(64, u, v, symmetric=False, self_loops=False)
    assert len(P.build_tiles(rp, c, 64, 500_000)["tile_col"]) == 1
    assert len(P.build_tiles(rp, c, 64, 500_001)["tile_col"]) == 0


def test_tau_zero_all_dense_and_tau_above_one_none():
    g = make_workload("c1", 0.1).graph
    a = P.build_tiles(g.rowptr, g.col, 64, 0)
    assert len(a["sp_col"]) == 0 and a["tile_nnz"].sum() == g.nnz
    b = P.build_tiles(g.rowptr, g.col, 64, 1_000_001)
    assert len(b["tile_col"]) == 0 and len(b["sp_col"]) == g.nnz
    np.testing.assert_array_equal(b["sp_rowptr"], g.rowptr)
    np.testing.assert_array_equal(b["sp_col"], g.col)


def test_empty_rows_and_ragged_tail():
    n, T = 200, 64  # 200 = 3*64 + 8: a ragged last tile
    u = np.array([0, 5, 199, 198, 130])
    v = np.array([199, 6, 199, 3, 131])
    rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    plan = P.build_tiles(rowptr, col, T, 100)
    R = 4
    assert len(plan["tile_rowptr"]) == R + 1
    # tile (3, 3) has area 8*8 = 64 and holds the (199, 199) edge: density 1/64 -> dense
    I = np.repeat(np.arange(R), np.diff(plan["tile_rowptr"]))
    assert (3, 3) in set(zip(I.tolist(), plan["tile_col"].tolist()))
