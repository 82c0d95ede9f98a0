"""Seeded synthetic inputs shared by the GPU path and the oracle.

This module holds no arithmetic of the scoring method: it only draws random
numbers and rounds them to the storage precision.  Every tensor is drawn from a
counter-based stream (numpy's Philox) keyed by ``(seed, tensor_id, chunk)``, so a
tensor's contents do not depend on the thread count or on the order in which
tensors are drawn, and large tensors can be drawn in parallel chunks.

bf16 tensors are returned as ``uint16`` bit patterns (round-to-nearest-even from
fp32); :func:`bf16_to_f64` widens them exactly.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 1 << 20  # elements per independent Philox stream


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _stream(seed: int, tensor_id: int, chunk: int) -> np.random.Generator:
    key = np.array([(int(seed) << 32) | (int(tensor_id) & 0xFFFFFFFF), int(chunk)],
                   dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest-even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    r = r.astype(np.uint16)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_to_f64(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64."""
    return bf16_to_f32(b).astype(np.float64)


def _fill(out: np.ndarray, seed: int, tensor_id: int, fn) -> None:
    flat = out.reshape(-1)
    n = flat.size
    nchunks = (n + CHUNK - 1) // CHUNK

    def work(c):
        lo = c * CHUNK
        hi = min(n, lo + CHUNK)
        flat[lo:hi] = fn(_stream(seed, tensor_id, c), hi - lo)

    if nchunks <= 1:
        for c in range(nchunks):
            work(c)
        return
    with ThreadPoolExecutor(max_workers=_threads()) as ex:
        list(ex.map(work, range(nchunks)))


def normal_f32(seed: int, tensor_id: int, shape, std: float = 1.0) -> np.ndarray:
    """N(0, std^2) drawn in fp32."""
    out = np.empty(shape, dtype=np.float32)
    s = np.float32(std)
    _fill(out, seed, tensor_id, lambda g, m: g.standard_normal(m, dtype=np.float32) * s)
    return out


def normal_bf16(seed: int, tensor_id: int, shape, std: float = 1.0) -> np.ndarray:
    """N(0, std^2) drawn in fp32 then rounded to bf16 (uint16 bit patterns)."""
    out = np.empty(shape, dtype=np.uint16)
    s = np.float32(std)
    _fill(out, seed, tensor_id,
          lambda g, m: f32_to_bf16_bits(g.standard_normal(m, dtype=np.float32) * s))
    return out


def uniform_ints(seed: int, tensor_id: int, shape, low: int, high: int) -> np.ndarray:
    """Integers uniform on [low, high) as int32."""
    out = np.empty(shape, dtype=np.int32)
    _fill(out, seed, tensor_id,
          lambda g, m: g.integers(low, high, size=m, dtype=np.int64).astype(np.int32))
    return out


def permutation(seed: int, tensor_id: int, n: int) -> np.ndarray:
    """A uniformly random permutation of 0..n-1 (int32)."""
    return _stream(seed, tensor_id, 0).permutation(n).astype(np.int32)
