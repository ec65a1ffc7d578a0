"""Seeded synthetic inputs shared by the CPU oracle tests and the HIP path.

This module holds no arithmetic of the method (no matmul, no convolution, no
gate math).  It only turns (seed, stream id, index) into numbers:

* SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014) used as a counter-based generator: element i of
  stream s under seed q is ``mix(s0 + (i + 1) * GAMMA)`` with
  ``s0 = q * 2**32 + s``.  For q = s = 0 this is exactly the published
  SplitMix64 sequence started from state 0.
* uniform(a, b): u = (x >> 40) * 2**-24 in [0, 1) (24 bits, exact in fp32),
  value = a + (b - a) * u computed in fp64, then rounded to fp32.
* normal: Box-Muller on two 53-bit uniforms from counters 2i and 2i+1,
  z = sqrt(-2 ln(1 - u1)) * cos(2 pi u2), computed in fp64, rounded to fp32.
* bf16: round-to-nearest-even of the fp32 bit pattern (what
  ``torch.Tensor.to(torch.bfloat16)`` does for finite values).
"""
from __future__ import annotations

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def _mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def splitmix64(seed: int, stream: int, n: int, start: int = 0) -> np.ndarray:
    """n consecutive 64-bit outputs of stream `stream`, beginning at counter `start`."""
    s0 = np.uint64((int(seed) << 32) + int(stream))
    i = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(s0 + i * GAMMA)


def _numel(shape) -> int:
    return int(np.prod(shape, dtype=np.int64)) if len(shape) else 1


def uniform(seed: int, stream: int, shape, lo: float, hi: float) -> np.ndarray:
    """fp32 array, i.i.d. uniform on [lo, hi)."""
    x = splitmix64(seed, stream, _numel(shape))
    u = (x >> np.uint64(40)).astype(np.float64) * (2.0 ** -24)
    return (lo + (hi - lo) * u).astype(np.float32).reshape(shape)


def normal(seed: int, stream: int, shape, scale: float = 1.0, mean: float = 0.0) -> np.ndarray:
    """fp32 array, i.i.d. normal(mean, scale**2) via Box-Muller."""
    n = _numel(shape)
    x = splitmix64(seed, stream, 2 * n)
    u = (x >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)
    u1, u2 = u[0::2], u[1::2]
    z = np.sqrt(-2.0 * np.log1p(-u1)) * np.cos(2.0 * np.pi * u2)
    return (mean + scale * z).astype(np.float32).reshape(shape)


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    with np.errstate(over="ignore"):
        return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> the fp32 values they denote (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 values rounded (RNE) to the nearest bf16, returned as fp32."""
    return bf16_bits_to_f32(to_bf16_bits(a))
