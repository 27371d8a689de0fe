"""Counter-based pseudo-random inputs that both the CPU and the GPU can
regenerate for any subset of rows, for inputs too large to build on the host
(the [E, F] edge features of the large graph).

value(row, f) depends only on (row, f, seed): the counter c = row * F + f is
split into 32-bit halves and mixed with the "lowbias32" integer hash
(x ^= x >> 16; x *= 0x7feb352d; x ^= x >> 15; x *= 0x846ca68b; x ^= x >> 16),
and the top 24 bits of the result give a float in [-1, 1) (exact in fp32).
Everything is int64 tensor arithmetic with no overflow (products are split
into 16-bit halves), so CPU and GPU produce identical bits. This module holds
no arithmetic of the method itself.
"""
from __future__ import annotations

import torch

_M32 = 0xFFFFFFFF


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2^32 for 0 <= x, c < 2^32, without int64 overflow."""
    lo = x * (c & 0xFFFF)
    hi = ((x * (c >> 16)) & 0xFFFF) << 16
    return (lo + hi) & _M32


def _lowbias32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    return x ^ (x >> 16)


def hashed_values(rows: torch.Tensor, F: int, seed: int = 0) -> torch.Tensor:
    """fp32 [len(rows), F] in [-1, 1) on rows.device; rows int64 >= 0."""
    rows = rows.to(torch.int64)
    f = torch.arange(F, dtype=torch.int64, device=rows.device)
    c = rows[:, None] * F + f[None, :]
    lo, hi = c & _M32, (c >> 32) & _M32
    x = _lowbias32(lo ^ _lowbias32((hi + (seed & _M32) * 0x9E37) & _M32))
    return (x >> 8).to(torch.float32) * (2.0 ** -23) - 1.0


def hashed_matrix(n: int, F: int, seed: int = 0, device="cpu", dtype=torch.float32, chunk: int = 1 << 22):
    """All rows 0 .. n-1, generated in chunks of rows (bounded temporaries)."""
    out = torch.empty((n, F), dtype=dtype, device=device)
    step = max(1, chunk // max(F, 1))
    for r0 in range(0, n, step):
        r1 = min(n, r0 + step)
        out[r0:r1] = hashed_values(torch.arange(r0, r1, dtype=torch.int64, device=device), F, seed).to(dtype)
    return out
