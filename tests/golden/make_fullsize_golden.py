"""Write the stored expected values of the full-size parity tests, from the oracle alone.

Run from the repository root:  python tests/golden/make_fullsize_golden.py [reorder] [dense]

* ``fullsize_reorder_plan.json``: for the 1M-node workloads c3 (power law) and c4 (block model), the oracle's
  cluster reordering (§3.3; 20 sweeps, seed 0, as the benchmark runs it), the relabelled CSR, and the tile plan
  (§3.4; 128-wide tiles at densities 1% and 5%) built on it.  Each array is stored as the SHA-256 of its
  little-endian bytes in a fixed integer type, plus a few sampled entries to name a mismatch.  The inputs'
  hashes are stored too, so a change of the generators shows as such.
* ``dense_c5_dkdv_cols.npz``: the full layer's dK and dV (§2.1 Eq. (1)) of 512 sampled columns at the 65,536 x
  8 x 64 workload, each column summed over all 65,536 rows with every row's softmax statistics (fp64, stored
  as fp32).

Nothing here calls the library: only ``oracle/`` and the seeded generators in ``synth/``.
"""

from __future__ import annotations

import hashlib
import json
import os
import sys
import time
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import attention as OA  # noqa: E402
from oracle import plan as OP  # noqa: E402
from oracle import reorder as OR  # noqa: E402
from synth import make_workload  # noqa: E402

REORDER_JSON = os.path.join(HERE, "fullsize_reorder_plan.json")
DENSE_NPZ = os.path.join(HERE, "dense_c5_dkdv_cols.npz")

ITERS, SEED, T = 20, 0, 128
TAUS = (10_000, 50_000)
# fixed integer type of each stored array
PLAN_TYPES = {"tile_rowptr": "<i8", "tile_col": "<i4", "tile_nnz": "<i4", "tile_mask": "<u4", "sp_rowptr": "<i8",
              "sp_col": "<i4", "sp_colptr": "<i8", "sp_row": "<i4", "tileT_ptr": "<i8", "tileT_idx": "<i4",
              "long_rows": "<i4", "long_cols": "<i4"}
DENSE_COLS = 512


def sha(x, dt: str) -> str:
    return hashlib.sha256(np.ascontiguousarray(x, dtype=np.dtype(dt)).tobytes()).hexdigest()


def samples(x, k: int = 16, seed: int = 0) -> dict:
    x = np.asarray(x)
    if x.size == 0:
        return {}
    pos = np.unique(np.concatenate([[0, x.size - 1], np.random.default_rng(seed).integers(0, x.size, k)]))
    return {str(int(p)): int(x.flat[p]) for p in pos}


def plan_arrays(rowptr, col, tau: int) -> dict:
    pl = OP.build_tiles(rowptr, col, T, tau)
    out = {k: pl[k] for k in PLAN_TYPES if k in pl}
    out["long_rows"] = np.flatnonzero(np.diff(pl["sp_rowptr"]) > 256)
    out["long_cols"] = np.flatnonzero(np.diff(pl["sp_colptr"]) > 256)
    return out


def reorder_record(name: str) -> dict:
    t0 = time.time()
    g = make_workload(name).graph
    labels, done = OR.lp_labels(g.rowptr, g.col, iters=ITERS, seed=SEED)
    perm, iperm = OR.cluster_order(g.rowptr, g.col, labels)
    rp2, cl2 = OP.permute_csr(g.rowptr, g.col, perm, iperm)
    rec = {
        "n": int(g.n), "nnz": int(g.nnz), "iters": ITERS, "seed": SEED, "sweeps_done": int(done),
        "input": {"rowptr": sha(g.rowptr, "<i8"), "col": sha(g.col, "<i4")},
        "labels": sha(labels, "<i4"), "perm": sha(perm, "<i4"), "iperm": sha(iperm, "<i4"),
        "perm_samples": samples(perm), "labels_samples": samples(labels, seed=1),
        "relabelled": {"rowptr": sha(rp2, "<i8"), "col": sha(cl2, "<i4")},
        "plans": {},
    }
    for tau in TAUS:
        arrs = plan_arrays(rp2, cl2, tau)
        rec["plans"][str(tau)] = {
            "T": T, "n_dense": int(len(arrs["tile_col"])), "nnz_sparse": int(len(arrs["sp_col"])),
            "sha256": {k: sha(v, PLAN_TYPES[k]) for k, v in arrs.items()},
        }
    print(f"{name}: n={g.n} nnz={g.nnz} sweeps={done} "
          f"dense={[rec['plans'][str(t)]['n_dense'] for t in TAUS]} ({time.time() - t0:.0f} s)", flush=True)
    return rec


def write_reorder():
    out = {"what": "oracle cluster order, relabelled CSR and tile plans at full size (see make_fullsize_golden.py)",
           "workloads": {name: reorder_record(name) for name in ("c3", "c4")}}
    with open(REORDER_JSON, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")


def _head_stats(args):
    q, k, v, do, scale = args
    return OA.dense_attn_row_stats(q, k, v, do, scale)


def write_dense():
    t0 = time.time()
    w = make_workload("c5")
    q, k, v, do = w.tensors()
    n, H, d = w.graph.n, w.heads, w.dim
    scale = 1.0 / np.sqrt(d)
    cols = np.unique(np.concatenate([[0, n - 1], np.random.default_rng(6).choice(n, DENSE_COLS - 2,
                                                                                  replace=False)]))
    # every row's (LSE, D), one head per process (the heads are independent)
    jobs = [tuple(np.ascontiguousarray(x[:, h:h + 1]) for x in (q, k, v, do)) + (scale,) for h in range(H)]
    with ProcessPoolExecutor(min(H, os.cpu_count() or 1)) as ex:
        per_head = list(ex.map(_head_stats, jobs))
    LSE = np.concatenate([s[0] for s in per_head], axis=1)
    Dv = np.concatenate([s[1] for s in per_head], axis=1)
    dK, dV = OA.dense_attn_dkdv_cols(q, k, v, do, scale, cols, stats=(LSE, Dv))
    inputs = hashlib.sha256(b"".join(np.ascontiguousarray(x, np.float32).tobytes() for x in (q, k, v, do)))
    np.savez_compressed(DENSE_NPZ, cols=cols.astype(np.int64), dK=dK.astype(np.float32),
                        dV=dV.astype(np.float32), inputs_sha256=np.array(inputs.hexdigest()))
    print(f"c5 dense: {len(cols)} columns ({time.time() - t0:.0f} s)", flush=True)


if __name__ == "__main__":
    which = set(sys.argv[1:]) or {"reorder", "dense"}
    if "dense" in which:
        write_dense()
    if "reorder" in which:
        write_reorder()
