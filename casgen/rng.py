"""Counter-based seeded random numbers for synthetic inputs.

This module is shared by the oracle-side tests and by the GPU-side tests and
bench: it produces the input bits that both sides receive. It holds none of
the attention arithmetic.

Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014). Its i-th output for state ``key`` is
``mix(key + (i + 1) * GOLDEN_GAMMA)``, so it is evaluated here as a pure
function of a counter, which vectorises in numpy. Independent substreams are
keyed by hashing a path of integers (config seed, tensor tag, batch row,
segment id, ...) through the same finaliser.

Normals: Box-Muller (Box and Muller, 1958) in float64 on consecutive pairs of
uniforms, both the cosine and the sine branch used.

Rounding: float64 -> float32 with numpy's round-to-nearest-even, then
float32 -> bfloat16 with round-to-nearest-even on the bit pattern.
"""
from __future__ import annotations

import numpy as np

GOLDEN_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_MASK64 = (1 << 64) - 1

# Tensor tags of the substreams.
TAG_Q = 1
TAG_K_CART = 2
TAG_V_CART = 3
TAG_K_SELF = 4
TAG_V_SELF = 5
TAG_DO = 6
TAG_LENGTHS = 7
TAG_SELECT = 8
TAG_GAPS = 9


def _mix_py(z: int) -> int:
    """SplitMix64 finaliser on a Python int (mod 2**64)."""
    z &= _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def stream_key(*path: int) -> int:
    """Key of the substream named by a path of non-negative integers."""
    k = 0x243F6A8885A308D3  # fractional digits of pi, an arbitrary start
    for p in path:
        k = _mix_py(k ^ _mix_py((int(p) + 0x9E3779B97F4A7C15) & _MASK64))
    return k


def _mix_np(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def raw_u64(key: int, n: int, start: int = 0) -> np.ndarray:
    """Outputs ``start .. start+n-1`` of SplitMix64 seeded with ``key``."""
    with np.errstate(over="ignore"):
        ctr = np.arange(start + 1, start + n + 1, dtype=np.uint64)
        return _mix_np(np.uint64(key) + ctr * GOLDEN_GAMMA)


def uniform(key: int, n: int) -> np.ndarray:
    """``n`` float64 uniforms in the open interval (0, 1)."""
    bits = raw_u64(key, n) >> np.uint64(11)
    return (bits.astype(np.float64) + 0.5) * (2.0 ** -53)


def _normal_chunk(key: int, p0: int, p1: int, n: int, std: float, out: np.ndarray) -> None:
    with np.errstate(over="ignore"):
        bits = raw_u64(key, 2 * (p1 - p0), start=2 * p0) >> np.uint64(11)
    u = (bits.astype(np.float64) + 0.5) * (2.0 ** -53)
    u1, u2 = u[0::2], u[1::2]
    r = np.sqrt(-2.0 * np.log(u1)) * std
    ang = 2.0 * np.pi * u2
    z = np.empty(2 * (p1 - p0), dtype=np.float64)
    z[0::2] = r * np.cos(ang)
    z[1::2] = r * np.sin(ang)
    lo = 2 * p0
    hi = min(n, 2 * p1)
    out[lo:hi] = z[: hi - lo]


_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        import concurrent.futures
        import os
        _POOL = concurrent.futures.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1))
    return _POOL


def normal(key: int, n: int, std: float = 1.0, chunk: int = 1 << 17) -> np.ndarray:
    """``n`` float64 draws from N(0, std^2) by Box-Muller (chunks evaluated on a
    thread pool; the values do not depend on the chunking)."""
    out = np.empty(n, dtype=np.float64)
    npairs = (n + 1) // 2
    spans = [(p0, min(npairs, p0 + chunk)) for p0 in range(0, npairs, chunk)]
    if len(spans) <= 1:
        for p0, p1 in spans:
            _normal_chunk(key, p0, p1, n, std, out)
        return out
    list(_pool().map(lambda s: _normal_chunk(key, s[0], s[1], n, std, out), spans))
    return out


def f64_to_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return ((b + bias) >> np.uint32(16)).astype(np.uint16)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    return f32_to_bf16_bits(f64_to_f32(x))


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bits (used to build oracle-side copies)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def randint(key: int, n: int, lo: int, hi: int) -> np.ndarray:
    """``n`` integers uniform on the inclusive range [lo, hi]."""
    u = uniform(key, n)
    return (lo + np.floor(u * (hi - lo + 1))).astype(np.int64)


def choose_distinct(key: int, pool: int, k: int) -> list:
    """``k`` distinct ids from ``range(pool)``, uniform without replacement,
    in draw order (a partial Fisher-Yates shuffle driven by the substream)."""
    perm = list(range(pool))
    u = uniform(key, k)
    for i in range(k):
        j = i + int(np.floor(u[i] * (pool - i)))
        perm[i], perm[j] = perm[j], perm[i]
    return perm[:k]
