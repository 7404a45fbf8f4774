"""Seeded synthetic inputs.

This module only draws random numbers and stores them; it holds none of the
partitioning method's arithmetic.  Tests, the benchmark and the CPU oracle's
callers all take their inputs from here, so the GPU library and the oracle
always see the same bits.

Recipe: numpy PCG64 seeded with ``SeedSequence([240111202, workload_id,
tensor_idx])``; ``standard_normal(float32)`` times ``scale`` (1/sqrt(fan_in)
for weights); bfloat16 tensors are then quantised once with round-to-nearest-
even.  Integer-valued variants draw uniformly from a small symmetric range so
that every product and sum is exact in float32.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

SEED_ROOT = 240111202


def rng(workload_id: int, tensor_idx: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [SEED_ROOT, int(workload_id), int(tensor_idx)])))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bfloat16 bit patterns (uint16).
    NaN/Inf never occur in these inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class HostTensor:
    """A synthetic tensor: ``values`` (float32, exactly the stored numbers) and
    the storage dtype ('bf16' or 'f32'); ``bits`` holds the bfloat16 patterns."""
    values: np.ndarray
    dtype: str
    bits: np.ndarray | None = None

    @property
    def shape(self):
        return self.values.shape

    def f64(self) -> np.ndarray:
        return self.values.astype(np.float64)

    def to_device(self, device="cuda"):
        import torch
        if self.dtype == "bf16":
            t = torch.from_numpy(np.ascontiguousarray(self.bits).view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(self.values))
        return t.to(device)


def _make(x32: np.ndarray, dtype: str) -> HostTensor:
    if dtype == "bf16":
        bits = bf16_bits(x32)
        return HostTensor(bf16_to_f32(bits).reshape(x32.shape), "bf16", bits.reshape(x32.shape))
    if dtype == "f32":
        return HostTensor(np.ascontiguousarray(x32, np.float32), "f32")
    raise ValueError(dtype)


def gaussian(workload_id: int, tensor_idx: int, shape, scale: float = 1.0,
             dtype: str = "bf16") -> HostTensor:
    x = rng(workload_id, tensor_idx).standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return _make(x, dtype)


def small_ints(workload_id: int, tensor_idx: int, shape, lo: int = -3, hi: int = 3,
               dtype: str = "bf16") -> HostTensor:
    """Integers uniform in [lo, hi] (exact in bf16 and f32)."""
    x = rng(workload_id, tensor_idx).integers(lo, hi + 1, size=shape).astype(np.float32)
    return _make(x, dtype)


def ones(shape, dtype: str = "f32") -> HostTensor:
    return _make(np.ones(shape, np.float32), dtype)


def row_scaled(t: HostTensor, factors) -> HostTensor:
    """t with row i multiplied by factors[i], stored again in t's dtype (a
    ramp of magnitudes along the rows, e.g. keys whose scores grow with
    their position)."""
    x = (t.values * np.asarray(factors, np.float32)[:, None]).astype(np.float32)
    return _make(x, t.dtype)


def transposed(t: HostTensor) -> HostTensor:
    """The same tensor stored transposed (a row-major copy of t.T)."""
    v = np.ascontiguousarray(t.values.T)
    b = None if t.bits is None else np.ascontiguousarray(t.bits.T)
    return HostTensor(v, t.dtype, b)
