"""Seeded dense tensors (Q, K, V, dO) and bfloat16 rounding.

Values are drawn fp32 ~ N(0, 1).  For bfloat16 workloads they are rounded to
the nearest bfloat16 (ties to even) before anything else sees them, so the
oracle (which upcasts exactly to fp64) and the GPU read the same numbers.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_CHUNK = 1 << 20  # values per independently seeded chunk


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 array -> uint16 bfloat16 bit patterns, round to nearest, ties to even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """uint16 bfloat16 bit patterns -> fp32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bfloat16 and return them as fp32."""
    return bf16_to_f32(bf16_bits(x))


def normal_tensor(shape, key, dtype: str) -> np.ndarray:
    """fp32 N(0,1) draws, rounded to bfloat16 when ``dtype == 'bf16'`` (returned as fp32 values).

    ``key`` is a tuple of integers.  The values are generated in chunks of 2^20,
    chunk c from PCG64 seeded with SeedSequence(key + (c,)), so the result does
    not depend on how many threads fill it.
    """
    if dtype not in ("f32", "bf16"):
        raise ValueError(dtype)
    out = np.empty(int(np.prod(shape)), dtype=np.float32)
    n_chunks = (out.size + _CHUNK - 1) // _CHUNK
    key = tuple(int(k) for k in key)

    def fill(c):
        part = out[c * _CHUNK:(c + 1) * _CHUNK]
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(key + (c,))))
        rng.standard_normal(out=part, dtype=np.float32)
        if dtype == "bf16":
            u = part.view(np.uint32)
            u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
            u &= np.uint32(0xFFFF0000)

    workers = max(1, min(16, os.cpu_count() or 1, n_chunks))
    if workers == 1:
        for c in range(n_chunks):
            fill(c)
    else:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(n_chunks)))
    return out.reshape(shape)
