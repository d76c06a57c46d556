"""Seeded synthetic inputs for alpha-entmax attention tests and benchmarks.

This module holds no part of the attention arithmetic: it only draws the
random Q, K, V, dO tensors both the GPU path and the CPU oracle consume, and
converts between float32 and bfloat16 bit patterns.

Recipe (the efficiency workloads of the paper's Sec. 4.1 are Gaussian
queries/keys with a query temperature; no dataset is involved):

* PCG64 streams seeded ``seed + 0`` (Q), ``+1`` (K), ``+2`` (V), ``+3`` (dO),
  standard normal draws in float32, laid out [B, H, n, d] (d fastest);
* Q is multiplied by the temperature ``c`` in float32 *before* rounding;
* bf16 tensors are then rounded float32 -> bfloat16 with round-to-nearest-even;
* the GPU receives those exact bits and the oracle receives the same values
  widened to float64.
"""
from __future__ import annotations

import numpy as np

SEED_BASE = 20250217


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 -> bfloat16 (round to nearest, ties to even); uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounding = 0x7FFF + ((u >> 16) & 1)
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


class Tensor:
    """One generated tensor: ``raw`` holds the bits handed to the GPU (uint16
    for bf16, float32 for fp32); ``f64()`` widens the same values to fp64."""

    def __init__(self, raw: np.ndarray, dtype: str):
        self.raw = raw
        self.dtype = dtype

    @property
    def shape(self):
        return self.raw.shape

    def f32(self) -> np.ndarray:
        return bf16_bits_to_f32(self.raw) if self.dtype == "bf16" else self.raw

    def f64(self) -> np.ndarray:
        return self.f32().astype(np.float64)


def normal(shape, seed: int, scale: float = 1.0, dtype: str = "bf16") -> Tensor:
    if dtype not in ("bf16", "f32"):
        raise ValueError("dtype must be 'bf16' or 'f32'")
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return Tensor(f32_to_bf16_bits(x) if dtype == "bf16" else x, dtype)


def attention_inputs(B: int, H: int, n: int, d: int, c: float = 1.0, dtype: str = "bf16",
                     seed: int = SEED_BASE, with_dout: bool = False) -> dict:
    """Q ~ c*N(0,1), K, V (and dO) ~ N(0,1), iid, [B, H, n, d]."""
    shape = (B, H, n, d)
    out = {"q": normal(shape, seed + 0, c, dtype),
           "k": normal(shape, seed + 1, 1.0, dtype),
           "v": normal(shape, seed + 2, 1.0, dtype)}
    if with_dout:
        out["dout"] = normal(shape, seed + 3, 1.0, dtype)
    return out
