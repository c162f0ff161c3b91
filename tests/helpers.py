"""Shared helpers of the GPU parity tests: device transfer and the tolerances.

Tolerances (per output tensor, elementwise):
* fp32: |x - r| <= 1e-5 |r| + 1e-5 rms(r)
* bf16 inputs with fp32 accumulation: |x - r| <= 2e-2 + 1e-2 |r|
where r is the fp64 oracle computed from the same (bf16-rounded) inputs.
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
    x, r = x[fin], r[fin]
    if r.size == 0:
        return
    if dtype == "f32":
        tol = 1e-5 * np.abs(r) + 1e-5 * np.sqrt(np.mean(r * r))
    else:
        tol = 2e-2 + 1e-2 * np.abs(r)
    err = np.abs(x - r)
    bad = err > tol
    if bad.any():
        k = int(np.argmax(err - tol))
        raise AssertionError(f"{name}: {int(bad.sum())}/{r.size} outside tolerance; worst |x-r|={err[k]:.3e} "
                             f"at r={r[k]:.4e} (tol {tol[k]:.3e})")
