"""Counter-based, device-independent random numbers for synthetic workloads.

Every value is a pure function of (seed, stream, element index), computed with
integer arithmetic that is exact in int64 on any torch device, followed by one
IEEE float32 multiply.  The same call therefore produces bit-identical tensors
on the CPU and on a GPU, so test inputs can be generated where they are needed
(device memory for the kernels, host memory for the CPU reference) without one
side depending on the other.

Integer hash: the 32-bit "lowbias32" mixer (xorshift-multiply, constants
0x7feb352d and 0x846ca68b, published by C. Wellons, "Prospecting for Hash
Functions", 2018).  Products are formed from 16-bit halves so no int64
intermediate ever exceeds 2**48.

Approximately normal values: the sum S of four independent uniform 16-bit
integers (Irwin-Hall with n=4, excess kurtosis -0.3) centred and scaled to the
requested standard deviation.  2*S - 4*65535 is an even integer of magnitude at
most 262140, exact in float32; the only rounding is the final float32 multiply,
then (optionally) torch's round-to-nearest-even cast to bfloat16.

This module holds no arithmetic of the decoding method itself.
"""
from __future__ import annotations

import math
import zlib

import torch

M32 = 0xFFFFFFFF
_C1 = 0x7FEB352D
_C2 = 0x846CA68B
# standard deviation of a sum of four uniform integers on [0, 65535]
_SIGMA_S4 = math.sqrt(4.0 * (65536.0 ** 2 - 1.0) / 12.0)
# elements per chunk when generating large tensors (bounds temporary memory)
CHUNK = 1 << 24


def stream_id(name: str) -> int:
    """Stable 32-bit id for a named random stream."""
    return zlib.crc32(name.encode("utf-8")) & M32


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2**32 for int64 x in [0, 2**32), without int64 overflow."""
    lo = x & 0xFFFF
    hi = x >> 16
    return ((lo * c) + (((hi * c) & 0xFFFF) << 16)) & M32


def hash32(x: torch.Tensor) -> torch.Tensor:
    """lowbias32 mixer on int64 tensors holding values in [0, 2**32)."""
    x = x ^ (x >> 16)
    x = _mul32(x, _C1)
    x = x ^ (x >> 15)
    x = _mul32(x, _C2)
    x = x ^ (x >> 16)
    return x


def _keys(seed: int, stream: int):
    k1 = (seed * 0x9E3779B1 + stream) & M32
    k2 = (stream * 0x85EBCA77 + seed + 0x27D4EB2F) & M32
    k3 = (k1 ^ (k2 * 0xC2B2AE3D)) & M32
    return k1, k2, k3


def _two_words(idx: torch.Tensor, seed: int, stream: int):
    """Two 32-bit words per element index (int64 tensor, values < 2**48)."""
    k1, k2, k3 = _keys(seed, stream)
    a = hash32((idx & M32) ^ k1)
    a = hash32(a ^ (idx >> 32) ^ k2)
    b = hash32(a ^ k3)
    return a, b


def normal_(out: torch.Tensor, seed: int, name: str, std: float,
            offset: int = 0) -> torch.Tensor:
    """Fill `out` (float32 or bfloat16, contiguous) with approximately N(0, std^2)
    values for elements offset .. offset + out.numel() - 1 of stream `name`."""
    assert out.is_contiguous()
    flat = out.view(-1)
    n = flat.numel()
    dev = out.device
    stream = stream_id(name)
    scale = torch.tensor(std / (2.0 * _SIGMA_S4), dtype=torch.float32, device=dev)
    for s in range(0, n, CHUNK):
        e = min(n, s + CHUNK)
        idx = torch.arange(offset + s, offset + e, dtype=torch.int64, device=dev)
        a, b = _two_words(idx, seed, stream)
        ssum = (a & 0xFFFF) + (a >> 16) + (b & 0xFFFF) + (b >> 16)
        v = (2 * ssum - 4 * 65535).to(torch.float32) * scale
        flat[s:e].copy_(v.to(out.dtype))
    return out


def normal(shape, seed: int, name: str, std: float, dtype=torch.float32,
           device="cpu") -> torch.Tensor:
    out = torch.empty(shape, dtype=dtype, device=device)
    return normal_(out, seed, name, std)


def randint(n: int, high: int, seed: int, name: str, device="cpu") -> torch.Tensor:
    """n integers uniform on [0, high) (high < 2**31), as int64."""
    idx = torch.arange(n, dtype=torch.int64, device=device)
    a, _ = _two_words(idx, seed, stream_id(name))
    return (a * high) >> 32
