"""Counter-based splitmix64 streams (Steele, Lea & Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014), vectorised with numpy.

Draw ``i`` of a stream is the splitmix64 output after ``i + 1`` increments of
the state, so any element of a stream can be computed without the ones before
it.  Streams are derived from a master seed and a stream id.  This module holds
no part of the codec's arithmetic; it only produces the seeded inputs (scans and
weights) that both the oracle and the GPU path consume.
"""
from __future__ import annotations

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def _mix(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def stream_base(seed: int, stream: int) -> np.uint64:
    """Initial state of sub-stream ``stream`` of master seed ``seed``."""
    with np.errstate(over="ignore"):
        s = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) * _GOLDEN + np.uint64(stream & 0xFFFFFFFF)
    return np.uint64(_mix(np.array([s], dtype=np.uint64))[0])


def u64(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Raw 64-bit draws ``start .. start+count-1`` of a sub-stream."""
    base = stream_base(seed, stream)
    idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        state = base + idx * _GOLDEN
    return _mix(state)


def uniform(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Uniform doubles in [0, 1) with 53 random bits."""
    return (u64(seed, stream, start, count) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def normal(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Standard normals by the Box-Muller transform, one pair of uniforms each
    (draws ``2i`` and ``2i+1`` of the stream give normal ``i``)."""
    u = uniform(seed, stream, 2 * start, 2 * count).reshape(count, 2)
    u1 = 1.0 - u[:, 0]                       # (0, 1]: log never sees 0
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u[:, 1])
