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


def grad_term_rms(rowptr, col, q, k, v, do, scale):
    """Root-mean-square size of one term of each fp32 gradient, over every (edge, head):
    scale |dP_ij| |K_j| for dQ_i, scale |dP_ij| |Q_i| for dK_j, |dO_i| for dV_j and |dP_ij| for
    dS_ij = P_ij (dP_ij - D_i) (P_ij <= 1).

    A gradient that is zero through exact cancellation (a row with one edge has dS = 0) still carries the fp32
    rounding of its terms, so on graphs where most rows cancel these are the floors rho to use instead of the
    result's own size."""
    rows = np.repeat(np.arange(len(rowptr) - 1), np.diff(rowptr))
    col = np.asarray(col, dtype=np.int64)
    if not len(col):
        return 0.0, 0.0, 0.0, 0.0
    q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
    dp = np.abs(np.einsum("ehc,ehc->eh", do[rows], v[col]))
    nk, nq, ndo = (np.linalg.norm(x, axis=-1) for x in (k[col], q[rows], do[rows]))
    rms = lambda t: float(np.sqrt(np.mean(t * t)))
    return rms(scale * dp * nk), rms(scale * dp * nq), rms(ndo), rms(dp)


# Elementwise figures of every fp32 comparison, reported at the end of the session (conftest): the largest
# |x - r| / (1e-5 |r| + 1e-5 rms(r)) (above 1 means the elementwise reading of the fp32 bar would fail there) and
# the largest |x - r| / |r| over entries with |r| >= rms(r).
FP32_ELEMENTWISE: list[tuple[str, float, float]] = []


def _record_fp32_elementwise(x: np.ndarray, r: np.ndarray, name: str) -> None:
    fin = np.isfinite(r)
    x, r = x[fin], r[fin]
    if r.size == 0:
        return
    rms = float(np.sqrt(np.mean(r * r)))
    err = np.abs(x - r)
    ratio = float(np.max(err / (1e-5 * np.abs(r) + 1e-5 * rms))) if rms > 0 else float(err.max() > 0) * np.inf
    big = np.abs(r) >= rms
    rel = float(np.max(err[big] / np.abs(r[big]))) if big.any() else 0.0
    import os

    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0].split("::")[-1]
    FP32_ELEMENTWISE.append((f"{test} {name}".strip(), ratio, rel))


def assert_close(x, r, dtype: str, name: str, rho: float | None = None):
    """``rho``: for fp32, a floor for the tolerance's scale: used in place of the RMS of the reference's vector
    norms ([n, H, d] tensors) or of 1 (per-entry values) when larger."""
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    assert x.shape == r.shape, (name, x.shape, r.shape)
    fin = np.isfinite(r)
    assert np.array_equal(np.isfinite(x), fin), f"{name}: non-finite pattern differs"
    assert np.array_equal(x[~fin], r[~fin]), f"{name}: infinite values differ"
    if dtype == "f32":
        _record_fp32_elementwise(x, r, name)
        if r.ndim == 3:  # [n, H, d]: normwise per (node, head)
            rn = np.linalg.norm(r, axis=-1)
            rho = max(np.sqrt(np.mean(rn * rn)) if rn.size else 0.0, rho or 0.0)
            err = np.linalg.norm(x - r, axis=-1)
            tol = 1e-5 * (rn + rho)
        else:
            x, r = x[fin], r[fin]
            err = np.abs(x - r)
            tol = 1e-5 * np.maximum(max(1.0, rho or 0.0), np.abs(r))
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
