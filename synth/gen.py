"""Counter-based seeded random numbers for the synthetic attention workloads.

This module only draws numbers. It holds none of the attention arithmetic:
no scores, no softmax, no value aggregation. Both the fp64 oracle (through the
tests) and the GPU path consume what it produces.

Generator (published definitions, written out here):

* ``key = SeedSequence([2603, 4427, config, tensor]).generate_state(1, uint64)``
  names one stream per (workload, tensor).
* The i-th 64-bit draw of a stream is the i-th output of SplitMix64 seeded with
  ``key`` (Steele, Lea and Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014; the finaliser constants are Vigna's):
  ``z = key + (i + 1) * 0x9E3779B97F4A7C15``, then
  ``z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
  z ^= z >> 31``.
  Every draw depends only on (key, i), so any slice of a tensor can be drawn on
  its own, on any device, with any thread count, and gives the same bits.
* Standard normals use the Box-Muller transform in fp64 on draws 2e and 2e+1:
  ``u1 = (d_{2e} >> 11) * 2^-53``, ``u2 = (d_{2e+1} >> 11) * 2^-53``,
  ``z = sqrt(-2 ln(1 - u1)) * cos(2 pi u2)``, rounded once to fp32.

The integer part is evaluated on int64 torch tensors (two's-complement wrap is
the uint64 arithmetic the definition asks for; logical right shifts are masked
arithmetic shifts).
"""
from __future__ import annotations

import math

import numpy as np
import torch

_GAMMA = 0x9E3779B97F4A7C15
_MIX1 = 0xBF58476D1CE4E5B9
_MIX2 = 0x94D049BB133111EB
_MASK64 = (1 << 64) - 1


def _s64(x: int) -> int:
    """Reinterpret an unsigned 64-bit value as a signed int64."""
    x &= _MASK64
    return x - (1 << 64) if x >= (1 << 63) else x


def _lsr(z: torch.Tensor, s: int) -> torch.Tensor:
    """Logical right shift of int64 bit patterns."""
    return (z >> s) & ((1 << (64 - s)) - 1)


def stream_key(config: int, tensor: int) -> int:
    """64-bit stream key for tensor ``tensor`` of workload ``config``."""
    st = np.random.SeedSequence([2603, 4427, int(config), int(tensor)]).generate_state(1, np.uint64)
    return int(st[0])


def splitmix64(key: int, counter: torch.Tensor) -> torch.Tensor:
    """SplitMix64 output number ``counter`` (int64 tensor) of the stream ``key``.

    Returns the 64-bit outputs as int64 bit patterns."""
    z = (counter + 1) * _s64(_GAMMA) + _s64(key)
    z = (z ^ _lsr(z, 30)) * _s64(_MIX1)
    z = (z ^ _lsr(z, 27)) * _s64(_MIX2)
    return z ^ _lsr(z, 31)


def uniform53(key: int, counter: torch.Tensor) -> torch.Tensor:
    """Uniform fp64 in [0, 1) from the top 53 bits of draw ``counter``."""
    return _lsr(splitmix64(key, counter), 11).to(torch.float64) * (2.0 ** -53)


def normal_at(key: int, index: torch.Tensor) -> torch.Tensor:
    """Standard normals (fp32) at flat element indices ``index`` of stream ``key``."""
    index = index.to(torch.int64)
    u1 = uniform53(key, 2 * index)
    u2 = uniform53(key, 2 * index + 1)
    z = torch.sqrt(-2.0 * torch.log1p(-u1)) * torch.cos((2.0 * math.pi) * u2)
    return z.to(torch.float32)


def normal(key: int, numel: int, device="cpu", chunk: int = 1 << 24) -> torch.Tensor:
    """``numel`` standard normals (fp32, flat) of stream ``key``, drawn in chunks."""
    out = torch.empty(numel, dtype=torch.float32, device=device)
    for s in range(0, numel, chunk):
        e = min(numel, s + chunk)
        idx = torch.arange(s, e, dtype=torch.int64, device=device)
        out[s:e] = normal_at(key, idx)
    return out


def uniform_int(key: int, n: int, high: int, device="cpu") -> torch.Tensor:
    """``n`` integers in [0, high) (multiply-shift of the top 32 bits; bias < 2^-32 * high)."""
    idx = torch.arange(n, dtype=torch.int64, device=device)
    top = _lsr(splitmix64(key, idx), 32)
    return (top * high) >> 32


def permutation(key: int, n: int) -> torch.Tensor:
    """A permutation of 0..n-1: argsort of n draws of the stream (ties broken by index)."""
    idx = torch.arange(n, dtype=torch.int64)
    draws = _lsr(splitmix64(key, idx), 1)  # non-negative 63-bit sort keys
    return torch.argsort(draws, stable=True)
