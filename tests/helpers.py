"""Shared helpers of the GPU parity tests: device transfer and the tolerances.

Tolerances, r being the fp64 oracle computed from the same (bf16-rounded) inputs:
* fp32, "1e-5 relative" read normwise: for every (node, head) output vector
  ||x - r||_2 <= 1e-5 (||r||_2 + rho), rho being the root-mean-square of the
  vector norms over the whole tensor; a scalar per (node, head) (LSE) must
  satisfy |x - r| <= 1e-5 max(1, |r|).  Elementwise relative error is not
  attainable in fp32 for entries that are sums of many cancelling terms, and a
  vector that is small only through cancellation carries the absolute error of
  terms of typical size, hence the rho floor.
* bf16 inputs with fp32 accumulation, elementwise: |x - r| <= 2e-2 + 1e-2 |r|.
"""

from __future__ import annotations

import numpy as np
import torch

from synth import bf16_bits


def dev_csr(rowptr, col):
    return (torch.from_numpy(np.ascontiguousarray(rowptr, dtype=np.int64)).cuda(),
            torch.from_numpy(np.ascontiguousarray(col, dtype=np.int32)).cuda())


def dev_feat(x: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        bits = bf16_bits(x).view(np.int16)
        return torch.from_numpy(np.ascontiguousarray(bits)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def host(x: torch.Tensor) -> np.ndarray:
    return x.float().cpu().numpy().astype(np.float64)


def assert_close(x, r, dtype: str, name: str):
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    assert x.shape == r.shape, (name, x.shape, r.shape)
    fin = np.isfinite(r)
    assert np.array_equal(np.isfinite(x), fin), f"{name}: non-finite pattern differs"
    assert np.array_equal(x[~fin], r[~fin]), f"{name}: infinite values differ"
    if dtype == "f32":
        if r.ndim == 3:  # [n, H, d]: normwise per (node, head)
            rn = np.linalg.norm(r, axis=-1)
            rho = np.sqrt(np.mean(rn * rn)) if rn.size else 0.0
            err = np.linalg.norm(x - r, axis=-1)
            tol = 1e-5 * (rn + rho)
        else:
            x, r = x[fin], r[fin]
            err = np.abs(x - r)
            tol = 1e-5 * np.maximum(1.0, np.abs(r))
    else:
        x, r = x[fin], r[fin]
        err = np.abs(x - r)
        tol = 2e-2 + 1e-2 * np.abs(r)
    if err.size == 0:
        return
    bad = err > tol
    if bad.any():
        k = np.unravel_index(int(np.argmax(err - tol)), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())}/{err.size} outside tolerance; worst error {err[k]:.3e} "
                             f"(tol {tol[k]:.3e}) at {k}")
