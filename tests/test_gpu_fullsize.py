"""Full-size parity against stored oracle results (written by tests/golden/make_fullsize_golden.py, which calls
only the oracle):

* the cluster order (§3.3), the relabelled CSR and the tile plans (§3.4) of the two 1M-node workloads, bit for
  bit, through the library's reorder -> relabel -> tile build exactly as the benchmark runs them (20 sweeps,
  seed 0, 128-wide tiles); attention alone cannot show a wrong order, since it is permutation-equivariant;
* the full layer's dK and dV (§2.1 Eq. (1)) at 65,536 x 8 x 64 on 512 sampled columns, each of which needs the
  softmax statistics of every row.
"""

import hashlib
import json
import os
import sys

import numpy as np
import pytest
import torch

from synth import make_workload
from tests.helpers import assert_close, dev_csr, dev_feat, host

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def sha(x: torch.Tensor | np.ndarray, dt: str) -> str:
    if isinstance(x, torch.Tensor):
        x = x.cpu().numpy()
    return hashlib.sha256(np.ascontiguousarray(x, dtype=np.dtype(dt)).tobytes()).hexdigest()


def first_difference(got: np.ndarray, samples: dict) -> str:
    bad = [(int(k), v, int(got.flat[int(k)])) for k, v in samples.items() if int(got.flat[int(k)]) != v]
    return f"sampled entries differing (position, oracle, library): {bad[:6]}" if bad else "sampled entries agree"


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_full_size_reorder_relabel_and_plans_bit_exact(gt, name):
    ref = json.load(open(os.path.join(GOLDEN, "fullsize_reorder_plan.json")))["workloads"][name]
    g = make_workload(name).graph
    assert (g.n, g.nnz) == (ref["n"], ref["nnz"])
    assert sha(g.rowptr, "<i8") == ref["input"]["rowptr"] and sha(g.col, "<i4") == ref["input"]["col"], \
        "the generator no longer gives the graph the stored results were computed on"
    say("full-size reorder", name, g.n, g.nnz)
    rp, cl = dev_csr(g.rowptr, g.col)
    perm, iperm, labels, sweeps = gt.reorder(rp, cl, iters=ref["iters"], seed=ref["seed"], want_sweeps=True)
    torch.cuda.synchronize()
    assert sweeps == ref["sweeps_done"]
    lab_h, perm_h = labels.cpu().numpy(), perm.cpu().numpy()
    assert sha(lab_h, "<i4") == ref["labels"], "labels: " + first_difference(lab_h, ref["labels_samples"])
    assert sha(perm_h, "<i4") == ref["perm"], "perm: " + first_difference(perm_h, ref["perm_samples"])
    assert sha(iperm, "<i4") == ref["iperm"]
    rp2, cl2 = gt.permute_csr(rp, cl, perm, iperm)
    assert sha(rp2, "<i8") == ref["relabelled"]["rowptr"] and sha(cl2, "<i4") == ref["relabelled"]["col"]
    for tau, pr in sorted(ref["plans"].items()):
        say("  plan", name, tau)
        plan = gt.build_tiles(rp2, cl2, pr["T"], int(tau))
        assert (plan.n_dense, plan.nnz_sparse) == (pr["n_dense"], pr["nnz_sparse"])
        got = plan.to_numpy()
        for key, want in pr["sha256"].items():
            x = got[key].view(np.uint32) if key == "tile_mask" else got[key]
            dt = "<u4" if key == "tile_mask" else ("<i8" if key.endswith("ptr") else "<i4")
            assert sha(x, dt) == want, f"{name} tau={tau}: {key}"


def test_dense_layer_65536_sampled_columns(gt):
    ref = np.load(os.path.join(GOLDEN, "dense_c5_dkdv_cols.npz"))
    w = make_workload("c5")
    n, H, d = w.graph.n, w.heads, w.dim
    q, k, v, do = w.tensors()
    digest = hashlib.sha256(b"".join(np.ascontiguousarray(x, np.float32).tobytes() for x in (q, k, v, do)))
    assert digest.hexdigest() == str(ref["inputs_sha256"]), \
        "the generator no longer gives the tensors the stored results were computed on"
    scale = 1.0 / np.sqrt(d)
    Q, K, V, dO = (dev_feat(x, "bf16") for x in (q, k, v, do))
    say("dense c5 sampled columns", n, H, d, len(ref["cols"]))
    O, L = gt.dense_attn_fwd(Q, K, V, scale)
    dQ, dK, dV = gt.dense_attn_bwd(Q, K, V, O, dO, L, scale)
    torch.cuda.synchronize()
    cols = torch.from_numpy(ref["cols"]).cuda()
    assert_close(host(dK[cols]), ref["dK"].astype(np.float64), "bf16", "dK columns")
    assert_close(host(dV[cols]), ref["dV"].astype(np.float64), "bf16", "dV columns")
