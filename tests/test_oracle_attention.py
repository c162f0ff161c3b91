"""Pins of the attention oracle against things other than itself.

* a dense masked softmax (a different formulation: an N x N score matrix with
  -inf outside the graph, scipy's softmax / logsumexp);
* the textbook full attention of §2.1 Eq. (1) as computed by torch's
  scaled_dot_product_attention in fp64;
* closed-form special cases (self-only rows, zero queries, all-ones values,
  a common shift of every key);
* permutation equivariance;
* torch fp64 autograd of the dense masked formulation, and central finite
  differences, for the backward;
* the sum rules sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i.
"""

import numpy as np
import pytest
import scipy.special
import torch

from oracle import attention as A
from synth import csr_from_pairs


def random_graph(n, p, seed, self_loops=True, symmetric=True, drop_rows=()):
    rng = np.random.default_rng(seed)
    m = rng.random((n, n)) < p
    np.fill_diagonal(m, False)
    u, v = np.nonzero(m)
    rowptr, col = csr_from_pairs(n, u, v, symmetric=symmetric, self_loops=self_loops)
    if drop_rows:
        dense = to_dense(rowptr, col, n)
        for r in drop_rows:
            dense[r, :] = False
        u, v = np.nonzero(dense)
        rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    return rowptr, col


def to_dense(rowptr, col, n):
    m = np.zeros((n, n), dtype=bool)
    for i in range(n):
        m[i, col[rowptr[i]:rowptr[i + 1]]] = True
    return m


def qkv(n, h, d, seed):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((n, h, d)) for _ in range(4)]


def masked_reference(mask, Q, K, V, scale):
    n, H, d = Q.shape
    O = np.zeros((n, H, d))
    L = np.full((n, H), -np.inf)
    for h in range(H):
        s = scale * Q[:, h, :] @ K[:, h, :].T
        s = np.where(mask, s, -np.inf)
        ok = mask.any(axis=1)
        p = np.zeros_like(s)
        p[ok] = scipy.special.softmax(s[ok], axis=1)
        O[:, h, :] = p @ V[:, h, :]
        L[ok, h] = scipy.special.logsumexp(s[ok], axis=1)
    return O, L


@pytest.mark.parametrize("seed", range(6))
def test_fwd_matches_dense_masked_softmax(seed):
    n = [7, 16, 33, 64, 50, 21][seed]
    rowptr, col = random_graph(n, 0.15, seed, symmetric=seed % 2 == 0, drop_rows=(2,) if seed > 2 else ())
    Q, K, V, _ = qkv(n, 3, 8, seed)
    scale = 0.37
    O, L = A.sparse_attn_fwd(rowptr, col, Q, K, V, scale)
    O_ref, L_ref = masked_reference(to_dense(rowptr, col, n), Q, K, V, scale)
    np.testing.assert_allclose(O, O_ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(np.isinf(L), np.isinf(L_ref))
    fin = np.isfinite(L_ref)
    np.testing.assert_allclose(L[fin], L_ref[fin], rtol=1e-12, atol=1e-12)


def test_complete_graph_is_eq1_torch_sdpa():
    n, H, d = 40, 2, 16
    rowptr = np.arange(0, n * n + 1, n, dtype=np.int64)
    col = np.tile(np.arange(n, dtype=np.int32), n)
    Q, K, V, _ = qkv(n, H, d, 11)
    O, _ = A.sparse_attn_fwd(rowptr, col, Q, K, V, 1.0 / np.sqrt(d))
    t = lambda x: torch.from_numpy(x).permute(1, 0, 2).contiguous()  # [H, N, d]
    ref = torch.nn.functional.scaled_dot_product_attention(t(Q), t(K), t(V)).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(O, ref, rtol=1e-12, atol=1e-12)
    O2, L2 = A.dense_attn_fwd(Q, K, V, 1.0 / np.sqrt(d))
    np.testing.assert_allclose(O2, ref, rtol=1e-12, atol=1e-12)
    _, L = A.sparse_attn_fwd(rowptr, col, Q, K, V, 1.0 / np.sqrt(d))
    np.testing.assert_allclose(L2, L, rtol=1e-12, atol=1e-12)


def test_weights_sum_to_one_via_constant_values():
    rowptr, col = random_graph(30, 0.2, 3, drop_rows=(5,))
    Q, K, _, _ = qkv(30, 2, 4, 3)
    V = np.ones((30, 2, 4))
    O, L = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.8)
    nonempty = np.diff(rowptr) > 0
    np.testing.assert_allclose(O[nonempty], 1.0, rtol=0, atol=1e-14)
    assert np.all(O[~nonempty] == 0) and np.all(np.isneginf(L[~nonempty]))


def test_self_only_row_and_zero_query():
    n = 12
    u = np.array([0, 0, 0, 1, 2, 3])
    v = np.array([1, 2, 3, 2, 3, 4])
    rowptr, col = csr_from_pairs(n, u, v, symmetric=True, self_loops=True)
    Q, K, V, _ = qkv(n, 2, 5, 4)
    O, _ = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.5)
    for i in range(5, n):  # isolated nodes: only the self-loop
        np.testing.assert_array_equal(O[i], V[i])
    O0, _ = A.sparse_attn_fwd(rowptr, col, np.zeros_like(Q), K, V, 0.5)
    for i in range(n):
        nb = col[rowptr[i]:rowptr[i + 1]]
        np.testing.assert_allclose(O0[i], V[nb].mean(axis=0), rtol=1e-13, atol=1e-14)


def test_common_key_shift_leaves_output_unchanged():
    rowptr, col = random_graph(25, 0.3, 8)
    Q, K, V, _ = qkv(25, 3, 6, 8)
    u = np.random.default_rng(1).standard_normal((1, 3, 6))
    O, L = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.7)
    O2, L2 = A.sparse_attn_fwd(rowptr, col, Q, K + u, V, 0.7)
    np.testing.assert_allclose(O2, O, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(L2, L + 0.7 * np.einsum("nhc,hc->nh", Q, u[0]), rtol=1e-11, atol=1e-11)


def test_permutation_equivariance():
    n = 45
    rowptr, col = random_graph(n, 0.12, 21, symmetric=False)
    Q, K, V, _ = qkv(n, 2, 8, 21)
    p = np.random.default_rng(5).permutation(n)  # new -> old
    ip = np.empty(n, np.int64)
    ip[p] = np.arange(n)
    dense = to_dense(rowptr, col, n)
    pd = dense[np.ix_(p, p)]
    u, v = np.nonzero(pd)
    rp2, c2 = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    O, L = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.3)
    O2, L2 = A.sparse_attn_fwd(rp2, c2, Q[p], K[p], V[p], 0.3)
    np.testing.assert_allclose(O2, O[p], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(L2, L[p], rtol=1e-12, atol=1e-13)


def torch_masked_grads(mask, Q, K, V, dO, scale):
    tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (Q, K, V))
    m = torch.tensor(mask)
    ok = m.any(dim=1)
    s = torch.einsum("ihc,jhc->hij", tq, tk) * scale
    s = s.masked_fill(~m[None], float("-inf"))
    s = torch.where(ok[None, :, None], s, torch.zeros_like(s))
    p = torch.softmax(s, dim=-1) * ok[None, :, None]
    o = torch.einsum("hij,jhc->ihc", p, tv)
    (o * torch.tensor(dO)).sum().backward()
    return tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


@pytest.mark.parametrize("seed", range(4))
def test_bwd_matches_torch_autograd(seed):
    n = [10, 24, 37, 60][seed]
    rowptr, col = random_graph(n, 0.18, 100 + seed, symmetric=seed % 2 == 1, drop_rows=(1,) if seed > 1 else ())
    Q, K, V, dO = qkv(n, 2, 8, 100 + seed)
    dQ, dK, dV = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.45)
    rq, rk, rv = torch_masked_grads(to_dense(rowptr, col, n), Q, K, V, dO, 0.45)
    np.testing.assert_allclose(dQ, rq, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dK, rk, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dV, rv, rtol=1e-11, atol=1e-12)


def test_bwd_central_finite_differences():
    n, H, d = 9, 2, 3
    rowptr, col = random_graph(n, 0.35, 77, symmetric=False)
    Q, K, V, dO = qkv(n, H, d, 77)
    scale = 0.9
    dQ, dK, dV = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, scale)

    def loss(q, k, v):
        return float((A.sparse_attn_fwd(rowptr, col, q, k, v, scale)[0] * dO).sum())

    eps = 1e-6
    rng = np.random.default_rng(0)
    for which, grad in ((0, dQ), (1, dK), (2, dV)):
        for _ in range(12):
            idx = tuple(rng.integers(0, s) for s in (n, H, d))
            args = [Q.copy(), K.copy(), V.copy()]
            args[which][idx] += eps
            up = loss(*args)
            args[which][idx] -= 2 * eps
            dn = loss(*args)
            assert abs((up - dn) / (2 * eps) - grad[idx]) < 1e-8


def test_bwd_sum_rules_and_self_only_row():
    n = 40
    rowptr, col = random_graph(n, 0.1, 9, symmetric=False, drop_rows=(3,))
    # make node 7 attend only to itself
    dense = to_dense(rowptr, col, n)
    dense[7, :] = False
    dense[7, 7] = True
    u, v = np.nonzero(dense)
    rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    Q, K, V, dO = qkv(n, 3, 5, 9)
    dQ, dK, dV = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.6)
    nonempty = np.diff(rowptr) > 0
    np.testing.assert_allclose(dK.sum(axis=0), 0.0, atol=1e-12)
    np.testing.assert_allclose(dV.sum(axis=0), dO[nonempty].sum(axis=0), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dQ[7], 0.0, atol=1e-15)
    assert np.all(dQ[3] == 0)


def test_bwd_sampled_equals_full():
    n = 70
    rowptr, col = random_graph(n, 0.08, 5, symmetric=False)
    Q, K, V, dO = qkv(n, 2, 4, 5)
    full = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.5)
    rows = np.array([0, 13, 69, 40])
    cols = np.array([2, 13, 68])
    dq, dk, dv = A.sparse_attn_bwd_sampled(rowptr, col, Q, K, V, dO, 0.5, rows, cols)
    np.testing.assert_allclose(dq, full[0][rows], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dk, full[1][cols], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dv, full[2][cols], rtol=1e-12, atol=1e-13)


def test_dense_bwd_matches_torch_and_sampled_rows():
    n, H, d = 48, 2, 8
    Q, K, V, dO = qkv(n, H, d, 31)
    scale = 1.0 / np.sqrt(d)
    dQ, dK, dV = A.dense_attn_bwd(Q, K, V, dO, scale)
    rq, rk, rv = torch_masked_grads(np.ones((n, n), bool), Q, K, V, dO, scale)
    np.testing.assert_allclose(dQ, rq, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dK, rk, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dV, rv, rtol=1e-11, atol=1e-12)
    rows = np.array([0, 5, 47])
    np.testing.assert_allclose(A.dense_attn_dq_rows(Q, K, V, dO, scale, rows), dQ[rows], rtol=1e-12, atol=1e-13)
    O, L = A.dense_attn_fwd(Q, K, V, scale, rows=rows)
    O_all, L_all = A.dense_attn_fwd(Q, K, V, scale)
    np.testing.assert_allclose(O, O_all[rows], rtol=1e-13)
    np.testing.assert_allclose(L, L_all[rows], rtol=1e-13)


def test_dense_sampled_columns_match_torch_autograd():
    # dK, dV of chosen columns (every row's softmax statistics needed) against torch's fp64 autograd of the
    # full layer, on a ragged column set in an order of its own, and with the statistics passed in
    n, H, d = 70, 3, 8
    Q, K, V, dO = qkv(n, H, d, 47)
    scale = 1.0 / np.sqrt(d)
    _, rk, rv = torch_masked_grads(np.ones((n, n), bool), Q, K, V, dO, scale)
    cols = np.array([69, 0, 33, 34, 7])
    dk, dv = A.dense_attn_dkdv_cols(Q, K, V, dO, scale, cols)
    np.testing.assert_allclose(dk, rk[cols], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv, rv[cols], rtol=1e-10, atol=1e-12)
    stats = A.dense_attn_row_stats(Q, K, V, dO, scale)
    dk2, dv2 = A.dense_attn_dkdv_cols(Q, K, V, dO, scale, np.arange(n), stats=stats)
    np.testing.assert_allclose(dk2, rk, rtol=1e-10, atol=1e-12)
    # softmax Jacobian sum rules over all columns: sum_j dK_j = 0, sum_j dV_j = sum_i dO_i
    np.testing.assert_allclose(dk2.sum(axis=0), 0.0, atol=1e-11)
    np.testing.assert_allclose(dv2.sum(axis=0), dO.sum(axis=0), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- per-edge bias (§2.1 Eq. (3), §3.3)

def dense_bias(rowptr, col, bias, n):
    """The [H, n, n] dense form of a per-edge bias (0 outside the graph; masked anyway)."""
    H = bias.shape[1]
    B = np.zeros((H, n, n))
    for i in range(n):
        for e in range(rowptr[i], rowptr[i + 1]):
            B[:, i, col[e]] = bias[e]
    return B


def test_bias_matches_torch_autograd_of_dense_masked_formulation():
    # a different formulation: dense scores + dense bias, -inf outside the graph, torch softmax and autograd
    n, H, d = 23, 2, 8
    rowptr, col = random_graph(n, 0.25, seed=41)
    Q, K, V, dO = qkv(n, H, d, seed=42)
    bias = np.random.default_rng(43).standard_normal((len(col), H))
    mask = torch.from_numpy(to_dense(rowptr, col, n))
    q, k, v = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (Q, K, V))
    b = torch.tensor(dense_bias(rowptr, col, bias, n), dtype=torch.float64, requires_grad=True)
    s = 0.3 * torch.einsum("ihc,jhc->hij", q, k) + b
    s = s.masked_fill(~mask, float("-inf"))
    o = torch.einsum("hij,jhc->ihc", torch.softmax(s, dim=-1), v)
    (o * torch.from_numpy(dO)).sum().backward()
    O, L = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.3, bias=bias)
    np.testing.assert_allclose(O, o.detach().numpy(), rtol=1e-12, atol=1e-12)
    dQ, dK, dV, dB = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.3, bias=bias)
    np.testing.assert_allclose(dQ, q.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dK, k.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dV, v.grad.numpy(), rtol=1e-10, atol=1e-12)
    gb = b.grad.numpy()
    for i in range(n):
        for e in range(rowptr[i], rowptr[i + 1]):
            np.testing.assert_allclose(dB[e], gb[:, i, col[e]], rtol=1e-10, atol=1e-12)


def test_bias_zero_is_the_plain_attention_and_row_constant_shifts_only_lse():
    n, H, d = 31, 3, 4
    rowptr, col = random_graph(n, 0.2, seed=44)
    Q, K, V, dO = qkv(n, H, d, seed=45)
    O0, L0 = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.5)
    g0 = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.5)
    zero = np.zeros((len(col), H))
    O1, L1 = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.5, bias=zero)
    assert np.array_equal(O0, O1) and np.array_equal(L0, L1)
    g1 = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.5, bias=zero)
    for a, b in zip(g0, g1[:3]):
        assert np.array_equal(a, b)
    # a constant per (row, head): softmax is shift invariant, LSE moves by the constant, dB sums to 0 per row
    c = np.random.default_rng(46).standard_normal((n, H))
    rows = np.repeat(np.arange(n), np.diff(rowptr))
    O2, L2 = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.5, bias=c[rows])
    np.testing.assert_allclose(O2, O0, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(L2, L0 + c, rtol=1e-12, atol=1e-12)
    dQ, dK, dV, dB = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.5, bias=c[rows])
    for a, b in zip(g0, (dQ, dK, dV)):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)
    row_sums = np.add.reduceat(dB, rowptr[:-1], axis=0)
    np.testing.assert_allclose(row_sums, 0.0, atol=1e-12)


def test_bias_minus_infinity_removes_the_edge():
    n, H, d = 27, 2, 6
    rowptr, col = random_graph(n, 0.3, seed=47)
    Q, K, V, dO = qkv(n, H, d, seed=48)
    rng = np.random.default_rng(49)
    rows = np.repeat(np.arange(n), np.diff(rowptr))
    cut = (rng.random(len(col)) < 0.3) & (rows != col)  # keep every self-loop
    bias = np.where(cut[:, None], -np.inf, 0.0) * np.ones((1, H))
    keep = ~cut
    u, v = rows[keep], col[keep]
    rp2, cl2 = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    O, L = A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.4, bias=bias)
    O2, L2 = A.sparse_attn_fwd(rp2, cl2, Q, K, V, 0.4)
    np.testing.assert_allclose(O, O2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(L, L2, rtol=1e-12, atol=1e-13)
    dQ, dK, dV, dB = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.4, bias=bias)
    for a, b in zip((dQ, dK, dV), A.sparse_attn_bwd(rp2, cl2, Q, K, V, dO, 0.4)):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)
    assert np.all(dB[cut] == 0.0)


def test_bias_gradient_central_finite_differences():
    n, H, d = 9, 1, 3
    rowptr, col = random_graph(n, 0.4, seed=50)
    Q, K, V, dO = qkv(n, H, d, seed=51)
    bias = np.random.default_rng(52).standard_normal((len(col), H))
    _, _, _, dB = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.7, bias=bias)
    eps = 1e-6
    for e in range(0, len(col), 3):
        bp, bm = bias.copy(), bias.copy()
        bp[e, 0] += eps
        bm[e, 0] -= eps
        lp = (A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.7, bias=bp)[0] * dO).sum()
        lm = (A.sparse_attn_fwd(rowptr, col, Q, K, V, 0.7, bias=bm)[0] * dO).sum()
        assert abs((lp - lm) / (2 * eps) - dB[e, 0]) < 1e-7


def test_bias_bwd_sampled_equals_full():
    n, H, d = 40, 2, 4
    rowptr, col = random_graph(n, 0.15, seed=53)
    Q, K, V, dO = qkv(n, H, d, seed=54)
    bias = np.random.default_rng(55).standard_normal((len(col), H))
    full = A.sparse_attn_bwd(rowptr, col, Q, K, V, dO, 0.6, bias=bias)
    rows = np.array([0, 5, 17, 39])
    dq, dk, dv, (pos, db) = A.sparse_attn_bwd_sampled(rowptr, col, Q, K, V, dO, 0.6, rows, rows, bias=bias)
    np.testing.assert_allclose(dq, full[0][rows], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dk, full[1][rows], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dv, full[2][rows], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(db, full[3][pos], rtol=1e-12, atol=1e-13)
