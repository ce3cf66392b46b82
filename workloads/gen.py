"""Seeded synthetic input generators.

This module produces the *inputs* of the sparse-embedding hot path (token ids,
per-token gradient rows, table weights, row-to-owner maps).  It holds none of
the method's arithmetic: nothing here gathers, coalesces, packs or updates.
Both the CPU oracle's tests and the GPU path's tests/bench draw their inputs
from here, so the two sides always see identical bytes.

Published definitions used:
  * SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
    generators", OOPSLA 2014), used counter-style: draw i of a stream with key
    k is mix64(k + (i + 1) * GAMMA).
  * Box-Muller transform (Box & Muller 1958) for normals, evaluated in fp64.
  * Bounded Zipf: P(id = k) proportional to (k + 1) ** -s for k in [0, V),
    sampled by inverse CDF (fp64 CDF, first index whose CDF exceeds u).
  * bfloat16 round-to-nearest-even of fp32 bit patterns.
"""
from __future__ import annotations

import ctypes
import functools
import os
import subprocess

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB

# Stream purposes (part of a stream's key).
PURPOSE_WEIGHTS = 1
PURPOSE_IDS = 2
PURPOSE_GRADS = 3
PURPOSE_NEXT_IDS = 4
PURPOSE_MISC = 5

_CHUNK = 1 << 22  # elements per vectorised block (bounds temporaries to ~100 MB)


def mix64_int(z: int) -> int:
    """SplitMix64 output function on a Python int (mod 2**64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * _M1) & MASK64
    z = ((z ^ (z >> 27)) * _M2) & MASK64
    return z ^ (z >> 31)


def splitmix64_sequence(seed: int, n: int) -> list[int]:
    """The sequential SplitMix64 generator: state += GAMMA, output mix64(state)."""
    out, s = [], seed & MASK64
    for _ in range(n):
        s = (s + GAMMA) & MASK64
        out.append(mix64_int(s))
    return out


def _mix64_arr(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(_M1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(_M2)
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int, step: int, purpose: int) -> int:
    """Key of the stream for (config seed, training step, purpose)."""
    return mix64_int(seed ^ mix64_int((purpose << 40) ^ (step & ((1 << 40) - 1)) ^ 0x5EED))


def draws_u64(key: int, start: int, n: int) -> np.ndarray:
    """Draws start .. start+n-1 of stream `key` (counter-based SplitMix64)."""
    i = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix64_arr(np.uint64(key) + i * np.uint64(GAMMA))


def uniform53(key: int, start: int, n: int) -> np.ndarray:
    """Uniform doubles in [0, 1) with 53 random bits."""
    return (draws_u64(key, start, n) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


_HERE = os.path.dirname(os.path.abspath(__file__))
_FAST_SRC = os.path.join(_HERE, "fastgen.c")
_FAST_LIB = os.path.join(_HERE, "libfastgen.so")
_fast = None


def build_fast(verbose: bool = False) -> str:
    """Compile fastgen.c (the compiled twin of normal_f32_reference)."""
    cmd = ["gcc", "-std=c99", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           "-o", _FAST_LIB + ".tmp", _FAST_SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(_FAST_LIB + ".tmp", _FAST_LIB)
    return _FAST_LIB


def _fast_lib():
    global _fast
    if _fast is None:
        if not os.path.exists(_FAST_LIB) or os.path.getmtime(_FAST_LIB) < os.path.getmtime(_FAST_SRC):
            build_fast()
        lib = ctypes.CDLL(_FAST_LIB)
        lib.wl_normal_f32.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p]
        lib.wl_normal_f32.restype = None
        _fast = lib
    return _fast


def normal_f32(key: int, n: int, sigma: float = 1.0) -> np.ndarray:
    """n normals N(0, sigma^2) by Box-Muller in fp64, cast to fp32 (compiled twin
    of normal_f32_reference; the two agree to within one fp32 ulp)."""
    out = np.empty(n, dtype=np.float32)
    if n:
        _fast_lib().wl_normal_f32(key & MASK64, n, float(sigma), out.ctypes.data_as(ctypes.c_void_p))
    return out


def normal_f32_reference(key: int, n: int, sigma: float = 1.0) -> np.ndarray:
    """n normals N(0, sigma^2) by Box-Muller in fp64, cast to fp32."""
    out = np.empty(n, dtype=np.float32)
    npairs = (n + 1) // 2
    for p0 in range(0, npairs, _CHUNK):
        p1 = min(npairs, p0 + _CHUNK)
        u = uniform53(key, 2 * p0, 2 * (p1 - p0))
        u1, u2 = u[0::2], u[1::2]
        r = np.sqrt(-2.0 * np.log1p(-u1))  # 1 - u1 in (0, 1]
        th = 2.0 * np.pi * u2
        z = np.empty(2 * (p1 - p0), dtype=np.float64)
        z[0::2] = r * np.cos(th)
        z[1::2] = r * np.sin(th)
        lo, hi = 2 * p0, min(n, 2 * p1)
        out[lo:hi] = (sigma * z[: hi - lo]).astype(np.float32)
    return out


@functools.lru_cache(maxsize=8)
def _zipf_cdf(V: int, s: float) -> np.ndarray:
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    cdf[-1] = 1.0
    return cdf


def zipf_pmf(V: int, s: float) -> np.ndarray:
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


def zipf_ids(key: int, n: int, V: int, s: float) -> np.ndarray:
    """n ids from the bounded Zipf(s) law over [0, V); id k has rank k + 1."""
    cdf = _zipf_cdf(V, s)
    u = uniform53(key, 0, n)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def uniform_ids(key: int, n: int, V: int) -> np.ndarray:
    """n ids uniform over [0, V)."""
    u = uniform53(key, 0, n)
    return np.minimum((u * V).astype(np.int64), V - 1).astype(np.int32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bit patterns (uint16), round to nearest, ties to even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = (b & 0x7FFFFFFF) > 0x7F800000
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    r[nan] = ((b[nan] >> 16) | 0x40).astype(np.uint16)  # keep NaN quiet
    return r


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> fp32 values (exact widening; for display/stats)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def owner_mod(V: int, P: int) -> np.ndarray:
    """row_owner[id] = id mod P."""
    return (np.arange(V, dtype=np.int64) % P).astype(np.int32)


def owner_range(V: int, P: int) -> np.ndarray:
    """Contiguous row ranges of ceil(V / P) rows: row_owner[id] = id // ceil(V / P)."""
    blk = -(-V // P)
    return (np.arange(V, dtype=np.int64) // blk).astype(np.int32)
