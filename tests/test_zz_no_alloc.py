"""The entry point that allocates nothing (gt_dense_attn_bwd_noalloc): called through the C ABI, its outputs
equal those of gt_dense_attn_bwd, the call with a caller workspace that it shares its kernels with, bit for bit;
on two calls in a row, the second with a smaller input, so that what the first left in the library's scratch
array cannot leak into the second."""

import sys

import numpy as np
import pytest
import torch

from synth.tensors import normal_tensor
from tests.helpers import dev_feat

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(n, H, d, dtype, seed):
    return [dev_feat(normal_tensor((n, H, d), (seed, n, t), dtype), dtype) for t in range(4)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_equals_workspace_call_twice(gt, dtype):
    # first a larger input (ragged: 5,000 rows), then a smaller one (777 rows, other heads and width)
    for n, H, d in ((5000, 8, 64), (777, 2, 32)):
        say("noalloc", dtype, n, H, d)
        Q, K, V, dO = _inputs(n, H, d, dtype, 7 + H)
        scale = 1.0 / np.sqrt(d)
        O, L = gt.dense_attn_fwd(Q, K, V, scale)
        ref = gt.dense_attn_bwd(Q, K, V, O, dO, L, scale)
        got = gt.dense_attn_bwd_noalloc(Q, K, V, O, dO, L, scale)
        torch.cuda.synchronize()
        for name, a, b in zip(("dQ", "dK", "dV"), got, ref):
            assert torch.equal(a, b), f"{name} differs from gt_dense_attn_bwd ({dtype}, n={n}, H={H}, d={d})"


def test_noalloc_full_size_then_small(gt):
    # the 65,536 x 8 x 64 layer (2 MiB of scratch), then a 300-node layer
    for n, H, d in ((65536, 8, 64), (300, 4, 64)):
        say("noalloc bf16", n, H, d)
        Q, K, V, dO = _inputs(n, H, d, "bf16", 3)
        O, L = gt.dense_attn_fwd(Q, K, V)
        ref = gt.dense_attn_bwd(Q, K, V, O, dO, L)
        got = gt.dense_attn_bwd_noalloc(Q, K, V, O, dO, L)
        torch.cuda.synchronize()
        for name, a, b in zip(("dQ", "dK", "dV"), got, ref):
            assert torch.equal(a, b), f"{name} differs from gt_dense_attn_bwd (n={n})"


def test_noalloc_rejects_sizes_above_its_scratch(gt):
    lib = gt.load_library()
    assert lib.gt_dense_attn_bwd_noalloc_max_bytes() == 64 << 20
    x = torch.empty(16, dtype=torch.bfloat16, device="cuda")
    L = torch.empty(16, dtype=torch.float32, device="cuda")
    n = (64 << 20) // (4 * 16) + 1  # n * H * 4 bytes one row above the 64 MiB array, H = 16
    st = lib.gt_dense_attn_bwd_noalloc(n, 16, 64, gt.GT_BF16, x.data_ptr(), x.data_ptr(), x.data_ptr(),
                                       x.data_ptr(), x.data_ptr(), L.data_ptr(), 0.125, x.data_ptr(), x.data_ptr(),
                                       x.data_ptr(), None)
    assert st == gt.GT_ERR_UNSUPPORTED
    assert b"64 MiB" in lib.gt_last_error()
