"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This module only draws random numbers and rounds them to a storage dtype.  It
holds none of the arithmetic of the primitive graphs (no operator, no
reduction, no contraction): both the oracle and the HIP path consume the exact
same dtype-rounded tensors from here, and nothing else is shared between them.

Recipe (one tensor per call): ``numpy.random.Generator(PCG64(seed))`` draws
float32 samples from the stated distribution, which are then rounded
round-to-nearest-even to the storage dtype (fp32 / fp16 / bf16).  The seed of
tensor ``t`` (1-based) of workload ``w`` (1-based) is ``1000*w + t``.
"""

from __future__ import annotations

import numpy as np

STORAGE_DTYPES = ("f32", "f16", "bf16")


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 with round-to-nearest-even.

    Returns the raw 16-bit patterns as ``uint16``.  NaN inputs keep a quiet NaN
    pattern; infinities stay infinities.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    if nan.any():
        rounded = rounded.copy()
        rounded[nan] = 0x7FC0
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_to_storage(x32: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to ``dtype`` and return the storage array.

    fp32 -> float32, fp16 -> float16 (NumPy's cast is RNE), bf16 -> uint16 bits.
    """
    x32 = np.asarray(x32, dtype=np.float32)
    if dtype == "f32":
        return x32.copy()
    if dtype == "f16":
        return x32.astype(np.float16)
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError(f"unknown storage dtype {dtype!r}")


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact up-cast of a storage array to float64."""
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    return np.asarray(a).astype(np.float64)


def draw(seed: int, shape, dist: str, a: float = 0.0, b: float = 1.0) -> np.ndarray:
    """Draw float32 samples.

    dist "normal":  a + b * N(0,1)  (mean a, standard deviation b)
    dist "uniform": U(a, b)
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = tuple(int(s) for s in shape)
    if dist == "normal":
        z = rng.standard_normal(size=shape, dtype=np.float32)
        return (np.float32(a) + np.float32(b) * z).astype(np.float32)
    if dist == "uniform":
        u = rng.random(size=shape, dtype=np.float32)
        return (np.float32(a) + np.float32(b - a) * u).astype(np.float32)
    raise ValueError(f"unknown distribution {dist!r}")


def make_tensor(seed: int, shape, dtype: str, dist: str, a: float = 0.0, b: float = 1.0):
    """One seeded input tensor in storage form (see ``round_to_storage``)."""
    return round_to_storage(draw(seed, shape, dist, a, b), dtype)


def make_inputs(specs):
    """Build every input of a workload.

    ``specs`` is a sequence of ``(name, seed, shape, dtype, dist, a, b)``.
    Returns ``{name: storage_array}`` in the order given.
    """
    out = {}
    for name, seed, shape, dtype, dist, a, b in specs:
        out[name] = make_tensor(seed, shape, dtype, dist, a, b)
    return out
