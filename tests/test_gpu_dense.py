"""GPU full softmax attention (§2.1 Eq. (1), the interleaved dense layer of
§3.2) vs the fp64 oracle: whole outputs at small n (ragged sizes included),
sampled rows plus sum rules at the 65,536-node workload."""

import sys

import numpy as np
import pytest
import torch

from oracle import attention as OA
from synth import make_workload
from synth.tensors import normal_tensor
from tests.helpers import assert_close, dev_feat, host

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("n,H,d,dtype", [(2, 1, 32, "f32"), (77, 2, 32, "f32"), (300, 1, 64, "f32"),
                                         (300, 8, 64, "bf16"), (1000, 4, 32, "bf16"), (4096, 8, 64, "bf16"),
                                         (129, 16, 64, "bf16")])
def test_dense_layer_full_outputs(gt, n, H, d, dtype):
    say("dense", n, H, d, dtype)
    q, k, v, do = (normal_tensor((n, H, d), (n, H, d, t), dtype) for t in range(4))
    scale = 1.0 / np.sqrt(d)
    Q, K, V, dO = (dev_feat(x, dtype) for x in (q, k, v, do))
    O, L = gt.dense_attn_fwd(Q, K, V, scale)
    dQ, dK, dV = gt.dense_attn_bwd(Q, K, V, O, dO, L, scale)
    torch.cuda.synchronize()
    O_ref, L_ref = OA.dense_attn_fwd(q, k, v, scale)
    ref = OA.dense_attn_bwd(q, k, v, do, scale)
    assert_close(host(O), O_ref, dtype, "O")
    assert_close(L.cpu().numpy(), L_ref, dtype, "LSE")
    for name, x, r in zip(("dQ", "dK", "dV"), (dQ, dK, dV), ref):
        assert_close(host(x), r, dtype, name)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dense_layer_single_node(gt, dtype):
    # one key: P = 1, so O = V, LSE = scale <q, k>, dV = dO, and dQ = dK = 0 up to rounding of the terms
    q, k, v, do = (normal_tensor((1, 4, 64), (1, t), dtype) for t in range(4))
    Q, K, V, dO = (dev_feat(x, dtype) for x in (q, k, v, do))
    O, L = gt.dense_attn_fwd(Q, K, V, 0.125)
    dQ, dK, dV = gt.dense_attn_bwd(Q, K, V, O, dO, L, 0.125)
    torch.cuda.synchronize()
    assert np.array_equal(host(O), v.astype(np.float64))
    np.testing.assert_allclose(L.cpu().numpy(), 0.125 * np.einsum("nhc,nhc->nh", q, k), rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(host(dV), do, rtol=1e-6 if dtype == "f32" else 0, atol=1e-6)
    term = 0.125 * np.abs(do).max() * np.abs(v).max() * max(np.abs(k).max(), np.abs(q).max())
    assert np.abs(host(dQ)).max() <= 1e-4 * term and np.abs(host(dK)).max() <= 1e-4 * term


def test_dense_layer_65536_sampled_rows_and_sum_rules(gt):
    # 1,024 sampled rows of O, LSE and dQ against the oracle (each needs only its own scores against all
    # keys); dK and dV, which need every row's softmax, are checked through the sum rules.
    w = make_workload("c5")
    n, H, d = w.graph.n, w.heads, w.dim
    q, k, v, do = w.tensors()
    scale = 1.0 / np.sqrt(d)
    Q, K, V, dO = (dev_feat(x, "bf16") for x in (q, k, v, do))
    say("dense c5 full size", n, H, d)
    O, L = gt.dense_attn_fwd(Q, K, V, scale)
    dQ, dK, dV = gt.dense_attn_bwd(Q, K, V, O, dO, L, scale)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(5).choice(n, size=1024, replace=False))
    O_ref, L_ref = OA.dense_attn_fwd(q, k, v, scale, rows=rows)
    dq_ref = OA.dense_attn_dq_rows(q, k, v, do, scale, rows)
    idx = torch.from_numpy(rows).cuda()
    assert_close(host(O[idx]), O_ref, "bf16", "O rows")
    assert_close(L[idx].cpu().numpy(), L_ref, "bf16", "LSE rows")
    assert_close(host(dQ[idx]), dq_ref, "bf16", "dQ rows")
    # sum rules of the softmax Jacobian: sum_j dK_j = 0, sum_j dV_j = sum_i dO_i (per head and feature);
    # allowance: bf16 output rounding of every summed entry (2^-8 relative) plus 1e-3.
    gk, gv = host(dK), host(dV)
    tol_k = 2.0 ** -8 * np.abs(gk).sum(axis=0) + 1e-3
    tol_v = 2.0 ** -8 * np.abs(gv).sum(axis=0) + 1e-3
    assert np.all(np.abs(gk.sum(axis=0)) <= tol_k)
    assert np.all(np.abs(gv.sum(axis=0) - do.astype(np.float64).sum(axis=0)) <= tol_v)
