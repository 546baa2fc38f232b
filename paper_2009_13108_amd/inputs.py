"""Seeded synthetic inputs shaped like the NITI experiments' workloads.

This module holds none of the method's arithmetic.  It only draws integers,
so that the HIP library and the CPU oracle can be fed identical bytes.  The
generator is SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014) evaluated on a counter, so a
tensor is a pure function of (seed, element index) and is stable across
numpy versions and machines.

Seeds follow ``base_seed(config, tensor_id) = 200913108 + 100 * config +
tensor_id``.  Value ranges are the workloads' (post-ReLU activations
U[0,127], weights and errors U[-127,127], 5-bit operands U[-15,15],
labels U{0..classes-1}, 8-bit pixels U[0,255]).
"""
from __future__ import annotations

import math

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_CHUNK = 1 << 24


def base_seed(config: int, tensor_id: int) -> int:
    return 200913108 + 100 * int(config) + int(tensor_id)


def _splitmix64(seed: int, start: int, n: int) -> np.ndarray:
    i = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + i * _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        z = z ^ (z >> np.uint64(31))
    return z


def _signed64(v: int) -> int:
    v &= 0xFFFFFFFFFFFFFFFF
    return v - (1 << 64) if v >= (1 << 63) else v


def _lsr(z, k: int):
    # logical right shift of an int64 torch tensor
    return (z >> k) & ((1 << (64 - k)) - 1)


def _uniform_int_torch(seed: int, shape, lo: int, hi: int, dtype, device):
    """The same stream as uniform_int, evaluated with torch int64 ops on
    `device` (wrapping multiplication, logical shifts by masking)."""
    import torch
    tdt = {np.int8: torch.int8, np.uint8: torch.uint8, np.int32: torch.int32,
           np.int64: torch.int64}[np.dtype(dtype).type]
    n = int(math.prod(shape))
    span = hi - lo + 1
    assert 0 < span < (1 << 31)
    out = torch.empty(n, dtype=tdt, device=device)
    g, m1, m2, sd = (_signed64(0x9E3779B97F4A7C15), _signed64(0xBF58476D1CE4E5B9),
                     _signed64(0x94D049BB133111EB), _signed64(seed))
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        z = torch.arange(s + 1, s + m + 1, dtype=torch.int64, device=device) * g + sd
        z = (z ^ _lsr(z, 30)) * m1
        z = (z ^ _lsr(z, 27)) * m2
        z = z ^ _lsr(z, 31)
        v = (_lsr(z, 32) * span) >> 32
        out[s:s + m] = (v + lo).to(tdt)
    return out.reshape(shape)


def uniform_int(seed: int, shape, lo: int, hi: int, dtype=np.int8, device=None):
    """Integers uniform on [lo, hi] (inclusive), as ``dtype``.  With a torch
    ``device`` the same values are produced there as a torch tensor."""
    shape = tuple(int(s) for s in (shape if isinstance(shape, (tuple, list)) else (shape,)))
    if device is not None:
        return _uniform_int_torch(seed, shape, lo, hi, dtype, device)
    n = int(math.prod(shape))
    span = np.uint64(hi - lo + 1)
    out = np.empty(n, dtype=dtype)
    for s in range(0, n, _CHUNK):
        m = min(_CHUNK, n - s)
        z = _splitmix64(seed, s, m)
        with np.errstate(over="ignore"):
            v = ((z >> np.uint64(32)) * span) >> np.uint64(32)
        out[s:s + m] = (v.astype(np.int64) + lo).astype(dtype)
    return out.reshape(shape)


def activations(seed, shape, device=None):
    """Post-ReLU int8 activations, U[0,127]."""
    return uniform_int(seed, shape, 0, 127, device=device)


def weights(seed, shape, device=None):
    """int8 weights, U[-127,127]."""
    return uniform_int(seed, shape, -127, 127, device=device)


def errors8(seed, shape, device=None):
    """int8 errors, U[-127,127]."""
    return uniform_int(seed, shape, -127, 127, device=device)


def errors5(seed, shape, device=None):
    """5-bit operands (sign + 4 bits), U[-15,15]."""
    return uniform_int(seed, shape, -15, 15, device=device)


def labels(seed, batch, classes, device=None):
    return uniform_int(seed, (batch,), 0, classes - 1, dtype=np.int32, device=device)


def pixels(seed, shape, device=None):
    """8-bit image pixels, U[0,255]."""
    return uniform_int(seed, shape, 0, 255, dtype=np.uint8, device=device)


def weight_exponent(fan_in: int) -> int:
    """Static weight exponent for U[-127,127] weights: the power of two nearest
    to sqrt(6 / fan_in) / 127 (a He-uniform style scale; ties toward -inf).
    Used only to seed the per-layer exponents of the synthetic networks."""
    v = math.log2(math.sqrt(6.0 / fan_in) / 127.0)
    return int(math.ceil(v - 0.5))
