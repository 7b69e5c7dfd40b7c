"""Counter-based random numbers for the synthetic DyNN workloads.

This module holds no part of the executed method: it only turns
(seed, stream name, counter) into numbers.  Both the CPU oracle and the
GPU path read the bytes it produces, so they see identical inputs.

Generator: SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014) used in counter mode: the i-th 64-bit draw
of a stream is mix(key + (i + 1) * gamma) with gamma = 0x9E3779B97F4A7C15.
Uniforms take the top 53 bits; normals use the Box-Muller transform on the
uniform pair (2i, 2i + 1).  Because every value depends only on its counter,
sample i of a batch is the same whatever the batch size.
"""

from __future__ import annotations

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def _mix(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int, name: str) -> np.uint64:
    """64-bit key of a named stream: FNV-1a over "seed:name", then mixed."""
    h = 0xCBF29CE484222325
    for byte in f"{seed}:{name}".encode():
        h ^= byte
        h = (h * 0x100000001B3) & 0xFFFFFFFFFFFFFFFF
    return _mix(np.array([h], dtype=np.uint64))[0]


def bits64(key: np.uint64, start: int, count: int) -> np.ndarray:
    ctr = np.arange(start, start + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(key + (ctr + np.uint64(1)) * _GAMMA)


def uniform(key: np.uint64, start: int, count: int) -> np.ndarray:
    """float64 uniforms in [0, 1) at counters start .. start+count-1."""
    return (bits64(key, start, count) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def normal(key: np.uint64, start: int, count: int) -> np.ndarray:
    """float64 standard normals; normal i uses uniform counters 2i and 2i+1."""
    u = uniform(key, 2 * start, 2 * count)
    u1, u2 = u[0::2], u[1::2]
    return np.sqrt(-2.0 * np.log1p(-u1)) * np.cos(2.0 * np.pi * u2)
