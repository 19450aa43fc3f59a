"""Seeded random numbers for the synthetic workloads.

This module is input generation only: it holds none of the attention or paging
arithmetic, so the oracle and the device path may both consume what it makes.

Every named stream is numpy's Philox-4x64 counter-based generator (Salmon,
Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011)
keyed by (base seed, stream id).  Normals come from numpy's ziggurat sampler in
float32; bf16 storage is round-to-nearest-even of that float32 value.  Values
are produced in fixed-size chunks into reused buffers, and a stream yields the
same sequence however it is chunked.
"""
from __future__ import annotations

import numpy as np

_CHUNK = 1 << 20


def generator(seed: int, stream: int) -> np.random.Generator:
    """An independent Philox stream for (seed, stream)."""
    key = np.array([seed & 0xFFFFFFFFFFFFFFFF, (0x5A17 << 32) | (stream & 0xFFFFFFFF)],
                   dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


def f32_to_bf16_bits(x: np.ndarray, out: np.ndarray | None = None) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns.

    Inputs are finite by construction, so there is no NaN special case.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).reshape(-1).view(np.uint32)
    t = np.right_shift(u, np.uint32(16))
    np.bitwise_and(t, np.uint32(1), out=t)
    np.add(t, np.uint32(0x7FFF), out=t)
    np.add(t, u, out=t)
    np.right_shift(t, np.uint32(16), out=t)
    if out is None:
        return t.astype(np.uint16).reshape(np.shape(x))
    out.reshape(-1)[:] = t
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(seed: int, stream: int, shape, std: float = 0.5) -> np.ndarray:
    """N(0, 1) * std rounded to bf16, as uint16 bit patterns of ``shape``."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    g = generator(seed, stream)
    buf = np.empty(min(n, _CHUNK) if n else 1, dtype=np.float32)
    s = np.float32(std)
    for a in range(0, n, _CHUNK):
        b = min(n, a + _CHUNK)
        v = buf[: b - a]
        g.standard_normal(out=v, dtype=np.float32)
        np.multiply(v, s, out=v)
        f32_to_bf16_bits(v, out=out[a:b])
    return out.reshape(shape)


def integers(seed: int, stream: int, n: int, lo: int, hi: int) -> np.ndarray:
    """n integers uniform in the inclusive range [lo, hi]."""
    return generator(seed, stream).integers(lo, hi + 1, size=n, dtype=np.int64)


def permutation(seed: int, stream: int, n: int) -> np.ndarray:
    """A seeded uniformly random permutation of 0..n-1 (int32)."""
    return generator(seed, stream).permutation(n).astype(np.int32)


def choice(seed: int, stream: int, n: int, k: int) -> np.ndarray:
    """k distinct integers from 0..n-1, ascending."""
    return np.sort(generator(seed, stream).choice(n, size=k, replace=False)).astype(np.int64)
