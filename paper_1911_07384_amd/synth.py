"""Seeded synthetic inputs shared by the HIP path's tests/bench and the oracle.

This module only draws numbers: it holds none of the training method's
arithmetic.  Every tensor is produced as IEEE binary16 values from a
counter-based generator whose definition is public, so the bytes do not
depend on numpy's own random streams:

* SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014): the i-th draw of a stream is the SplitMix64
  output function applied to ``base + (i + 1) * 0x9E3779B97F4A7C15``.
* A stream's ``base`` is the SplitMix64 output of
  ``seed ^ (stream * 0xD1B54A32D192ED03)``, so every tensor of a workload has
  its own independent stream id.
* Uniforms on [0, 1) take the top 53 bits: ``(z >> 11) * 2**-53``.
* Normals come from the Box-Muller transform on consecutive uniform pairs
  (Box and Muller, 1958), in float64, then scaled by the standard deviation.
* Conversion to binary16 is numpy's ``astype(float16)`` (round to nearest,
  ties to even, directly from float64).
"""

from __future__ import annotations

import math

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_STREAM_MUL = 0xD1B54A32D192ED03
_MASK64 = (1 << 64) - 1


def _mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def _base(seed: int, stream: int) -> np.uint64:
    s = (int(seed) ^ ((int(stream) * _STREAM_MUL) & _MASK64)) & _MASK64
    with np.errstate(over="ignore"):
        return _mix(np.array([s], dtype=np.uint64) + _GAMMA)[0]


def raw_u64(n: int, seed: int, stream: int) -> np.ndarray:
    """The first ``n`` 64-bit outputs of stream ``stream`` of generator ``seed``."""
    base = _base(seed, stream)
    with np.errstate(over="ignore"):
        ctr = np.arange(1, n + 1, dtype=np.uint64)
        return _mix(base + ctr * _GAMMA)


def uniform(n: int, seed: int, stream: int) -> np.ndarray:
    """``n`` float64 uniforms on [0, 1)."""
    z = raw_u64(n, seed, stream)
    return (z >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def normal(n: int, seed: int, stream: int) -> np.ndarray:
    """``n`` float64 standard normals (Box-Muller on uniform pairs)."""
    m = (n + 1) // 2
    u = uniform(2 * m, seed, stream)
    u1, u2 = u[0::2], u[1::2]
    r = np.sqrt(-2.0 * np.log1p(-u1))
    th = 2.0 * math.pi * u2
    out = np.empty(2 * m, dtype=np.float64)
    out[0::2] = r * np.cos(th)
    out[1::2] = r * np.sin(th)
    return out[:n]


def normal_f16(shape, std: float, seed: int, stream: int, mean: float = 0.0) -> np.ndarray:
    """binary16 tensor with entries ~ N(mean, std^2), rounded to nearest even."""
    n = int(np.prod(shape)) if len(shape) else 1
    v = normal(n, seed, stream) * float(std) + float(mean)
    return v.astype(np.float16).reshape(shape)


def loguniform_f16(shape, lo_exp: float, hi_exp: float, seed: int, stream: int) -> np.ndarray:
    """binary16 tensor with |v| = 2**(lo + (hi - lo) * u) and an independent random sign."""
    n = int(np.prod(shape))
    z = raw_u64(n, seed, stream)
    u = (z >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)
    sign = np.where((z & np.uint64(1)) == np.uint64(1), -1.0, 1.0)
    v = sign * np.exp2(lo_exp + (hi_exp - lo_exp) * u)
    return v.astype(np.float16).reshape(shape)


def labels(n: int, classes: int, seed: int, stream: int) -> np.ndarray:
    """``n`` int32 labels uniform on [0, classes) by multiply-shift of the top 32 bits."""
    z = raw_u64(n, seed, stream) >> np.uint64(32)
    return ((z * np.uint64(classes)) >> np.uint64(32)).astype(np.int32)


def he_std(fan_in: int) -> float:
    """He-normal standard deviation sqrt(2 / fan_in) with fan_in = C*R*S."""
    return math.sqrt(2.0 / fan_in)


def bits(a: np.ndarray) -> np.ndarray:
    """View a float16 array as its uint16 bit patterns (no copy)."""
    return np.ascontiguousarray(a).view(np.uint16)
