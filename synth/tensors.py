"""Seeded dense tensors (Q, K, V, dO) and bfloat16 rounding.

Values are drawn fp32 ~ N(0, 1).  For bfloat16 workloads they are rounded to
the nearest bfloat16 (ties to even) before anything else sees them, so the
oracle (which upcasts exactly to fp64) and the GPU read the same numbers.
"""

from __future__ import annotations

import numpy as np


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


def normal_tensor(shape, rng: np.random.Generator, dtype: str) -> np.ndarray:
    """fp32 N(0,1) draws, rounded to bfloat16 when ``dtype == 'bf16'`` (returned as fp32 values)."""
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if dtype == "bf16":
        x = bf16_round(x)
    elif dtype != "f32":
        raise ValueError(dtype)
    return x
