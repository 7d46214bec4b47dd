"""Seeded synthetic inputs for the keyless-attention workloads.

This module only draws numbers. It holds none of the attention arithmetic: it
is shared by the CPU oracle side (tests, baseline timing) and the HIP side
(tests, bench) so that both consume identical input bits.

Generator (our own recipe, counter based so any slice can be drawn on any
device without drawing what precedes it):

* A 32-bit integer hash (Wellons' "lowbias32": xorshift 16, multiply by
  0x7feb352d, xorshift 15, multiply by 0x846ca68b, xorshift 16) is applied
  twice to a 32-bit counter mixed with two keys derived from ``(seed, stream)``.
  The hash is a bijection on 32-bit words, so distinct counters give distinct
  words.
* Element ``i`` of a tensor uses counters ``2i`` and ``2i+1`` for two uniforms
  ``u = (h + 0.5) / 2^32`` and one Box-Muller normal
  ``z = sqrt(-2 ln u1) cos(2 pi u2)`` in float64, scaled by ``std``, rounded to
  float32 (round to nearest even), then to bfloat16 (round to nearest even)
  when a bf16 tensor is requested.
* Integers (cache lengths) use ``lo + (h mod span)``; permutations sort by hash.

All integer steps are exact in int64 (a 32x32-bit product is split in 16-bit
halves so nothing overflows), so CPU and GPU give the same words. The float64
log/cos may differ in the last ulp between devices, which can move a value by
one float32 ulp; the oracle is always fed the bits that the GPU actually read
(copied back from device memory), so parity never depends on this.
"""

from __future__ import annotations

import math

import torch

_M32 = 0xFFFFFFFF
# Counters per draw are 32-bit; larger tensors are drawn in 2^31-element
# windows, each with its own derived stream key.
_WINDOW = 1 << 31
_CHUNK = 1 << 24


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2^32 for x in [0, 2^32) without int64 overflow."""
    lo = x & 0xFFFF
    hi = x >> 16
    return (lo * c + ((hi * c) & 0xFFFF) * 65536) & _M32


def _hash32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def _key(seed: int, stream: int, window: int = 0) -> tuple[int, int]:
    t = torch.tensor([(seed * 0x9E3779B9 + 0x632BE5AB) & _M32], dtype=torch.int64)
    k0 = _hash32(t)
    k1 = _hash32(k0 ^ ((stream * 0x85EBCA6B + window * 0xC2B2AE35 + 1) & _M32))
    return int(k0.item()), int(k1.item())


def _words(counter: torch.Tensor, k0: int, k1: int) -> torch.Tensor:
    return _hash32(_hash32(counter ^ k0) ^ k1)


def _normal_f64(start: int, count: int, k0: int, k1: int, device) -> torch.Tensor:
    idx = torch.arange(start, start + count, dtype=torch.int64, device=device)
    h1 = _words((2 * idx) & _M32, k0, k1)
    h2 = _words((2 * idx + 1) & _M32, k0, k1)
    u1 = (h1.to(torch.float64) + 0.5) * (1.0 / 4294967296.0)
    u2 = (h2.to(torch.float64) + 0.5) * (1.0 / 4294967296.0)
    return torch.sqrt(-2.0 * torch.log(u1)) * torch.cos((2.0 * math.pi) * u2)


def normal(shape, seed: int, stream: int, std: float = 1.0,
           dtype: torch.dtype = torch.bfloat16, device="cpu") -> torch.Tensor:
    """Tensor of ``shape`` with N(0, std^2) entries, as described above."""
    shape = tuple(int(s) for s in shape)
    n = math.prod(shape)
    out = torch.empty(n, dtype=dtype, device=device)
    pos = 0
    while pos < n:
        window = pos // _WINDOW
        k0, k1 = _key(seed, stream, window)
        take = min(_CHUNK, n - pos, (window + 1) * _WINDOW - pos)
        z = _normal_f64(pos - window * _WINDOW, take, k0, k1, device)
        z32 = (z * std).to(torch.float32)
        out[pos:pos + take] = z32.to(dtype)
        pos += take
    return out.view(shape)


def uniform_int(count: int, lo: int, hi: int, seed: int, stream: int) -> torch.Tensor:
    """``count`` integers uniform in [lo, hi] (inclusive), int64 on the CPU."""
    k0, k1 = _key(seed, stream)
    h = _words(torch.arange(count, dtype=torch.int64) & _M32, k0, k1)
    return lo + (h % (hi - lo + 1))


def permutation(n: int, seed: int, stream: int) -> torch.Tensor:
    """A random permutation of range(n) (int64, CPU): sort by hashed counter."""
    k0, k1 = _key(seed, stream)
    h = _words(torch.arange(n, dtype=torch.int64) & _M32, k0, k1)
    return torch.argsort(h)
