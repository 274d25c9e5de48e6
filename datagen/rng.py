"""Counter-based random streams for the synthetic workloads.

SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014) is applied to a counter, so element ``i`` of a
stream depends only on ``(key, i)``.  Any slice of any stream can be
regenerated on its own, on the CPU or on a GPU, with identical integer bits.

All arithmetic is done in torch ``int64`` tensors; multiplication wraps
modulo 2**64 exactly like ``uint64`` (two's complement), and logical right
shifts are emulated with a mask.  Uniforms take the top 53 bits; normals use
the Box-Muller transform in float64.

This module holds no part of the selective-transfer method: it only makes
inputs.  Tests, the bench and the oracle harness all draw from it.
"""
from __future__ import annotations

import math

import torch

_GAMMA = 0x9E3779B97F4A7C15
_MUL1 = 0xBF58476D1CE4E5B9
_MUL2 = 0x94D049BB133111EB


def _s64(x: int) -> int:
    """Reinterpret an unsigned 64-bit integer as a signed one."""
    x &= (1 << 64) - 1
    return x - (1 << 64) if x >= (1 << 63) else x


def _srl(x: torch.Tensor, s: int) -> torch.Tensor:
    """Logical right shift of int64 bit patterns."""
    return (x >> s) & ((1 << (64 - s)) - 1)


def mix64(x: torch.Tensor) -> torch.Tensor:
    """SplitMix64 output function on int64 bit patterns (wrapping)."""
    z = x + _s64(_GAMMA)
    z = (z ^ _srl(z, 30)) * _s64(_MUL1)
    z = (z ^ _srl(z, 27)) * _s64(_MUL2)
    return z ^ _srl(z, 31)


def mix64_int(x: int) -> int:
    """Python-int SplitMix64 output function (used to derive stream keys)."""
    z = (x + _GAMMA) & ((1 << 64) - 1)
    z = ((z ^ (z >> 30)) * _MUL1) & ((1 << 64) - 1)
    z = ((z ^ (z >> 27)) * _MUL2) & ((1 << 64) - 1)
    return z ^ (z >> 31)


def stream_key(*parts: int) -> int:
    """Fold a tuple of non-negative ints (seed, tag, request, layer, ...) into a key."""
    k = 0x5DEECE66D
    for p in parts:
        k = mix64_int(k ^ (int(p) & ((1 << 64) - 1)))
    return k


def raw64(key: int, count: int, device="cpu", start: int = 0) -> torch.Tensor:
    """``count`` int64 words of stream ``key`` starting at counter ``start``."""
    ctr = torch.arange(start, start + count, dtype=torch.int64, device=device)
    # the standard SplitMix64 sequence seeded with ``key``: state_i = key + i*gamma
    return mix64(ctr * _s64(_GAMMA) + _s64(key))


def uniform(key: int, count: int, device="cpu", start: int = 0) -> torch.Tensor:
    """Float64 uniforms in the open interval (0, 1)."""
    r = _srl(raw64(key, count, device, start), 11)
    return (r.to(torch.float64) + 0.5) * (1.0 / (1 << 53))


def normal(key: int, count: int, device="cpu", start: int = 0) -> torch.Tensor:
    """Float64 standard normals, one Box-Muller pair per output element.

    Element ``i`` of the stream uses uniforms ``2i`` and ``2i + 1``, so a slice
    starting at ``start`` equals the same slice of the full stream.
    """
    u = uniform(key, 2 * count, device, 2 * start).view(count, 2)
    return torch.sqrt(-2.0 * torch.log(u[:, 0])) * torch.cos((2.0 * math.pi) * u[:, 1])


def choice_without_replacement(key: int, lo: int, hi: int, n: int, device="cpu") -> torch.Tensor:
    """``n`` distinct integers drawn uniformly from ``[lo, hi)``, ascending."""
    if n == 0:
        return torch.empty(0, dtype=torch.int64, device=device)
    if n > hi - lo:
        raise ValueError("cannot draw more distinct values than the range holds")
    r = raw64(key, hi - lo, device)
    # the n smallest random keys pick a uniform n-subset; ties have
    # probability ~2^-64 and are broken by position (stable sort)
    order = torch.argsort(r, stable=True)[:n]
    return torch.sort(order + lo).values
