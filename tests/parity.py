"""Comparison helpers for GPU-vs-oracle parity (the tolerance rules).

  sum / mean : |gpu - ref| <= 1e-5 * S + 1e-6 in fp32, with ref the fp64
               oracle and S = sum |message| (per degree for mean);
               bf16 storage adds 1e-2 * |ref| (one bf16 rounding of the fp32
               accumulator is at most 2^-9 relative).
  max        : values bit-exact (bf16: the RNE rounding of the oracle's fp32
               maximum), argmax bit-exact.
  integers   : bit-exact.
  softmax    : |gpu - ref| <= ref * (1e-5 + 4 eps (|s| + |m| + 1)) + 1e-30,
               eps = 2^-24, s the edge's score and m its segment's maximum:
               the denominator is a sum of positive terms held to the 1e-5
               sum rule, and rounding s - m (or forming s in fp32) moves
               exp(s - m) by at most eps (|s| + |m|) relative.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle


def to_dev(a, dev="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def bf16_round(x_np: np.ndarray) -> np.ndarray:
    """fp32 values after a round trip through bf16 (RNE), as fp32."""
    return torch.from_numpy(np.ascontiguousarray(x_np, np.float32)).to(torch.bfloat16).float().numpy()


def check_sum(gpu: torch.Tensor, ref: np.ndarray, sabs: np.ndarray, bf16: bool = False, what: str = ""):
    g = gpu.float().cpu().numpy().astype(np.float64)
    bound = 1e-5 * sabs + 1e-6 + (1e-2 * np.abs(ref) if bf16 else 0.0)
    err = np.abs(g - ref)
    bad = err > bound
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} elements out of tolerance; first {tuple(i)} gpu={g[tuple(i)]!r} "
                             f"ref={ref[tuple(i)]!r} bound={bound[tuple(i)]!r}")
    return float((err / bound).max()) if err.size else 0.0


def check_max(gpu: torch.Tensor, garg: torch.Tensor, ref: np.ndarray, rarg: np.ndarray, bf16: bool = False, what: str = ""):
    want = ref.astype(np.float32)
    if bf16:
        want_t = torch.from_numpy(want).to(torch.bfloat16)
        got_t = gpu.cpu()
        ok = torch.equal(got_t.view(torch.int16), want_t.view(torch.int16))
    else:
        got = gpu.cpu().numpy()
        ok = np.array_equal(got.view(np.uint32), want.view(np.uint32))
    if not ok:
        g = gpu.float().cpu().numpy()
        bad = np.argwhere(g != want.astype(np.float32) if not bf16 else g != bf16_round(want))
        i = tuple(bad[0]) if bad.size else None
        raise AssertionError(f"{what}: max values differ (first {i}: gpu={g[i] if i else None} ref={want[i] if i else None})")
    a = garg.cpu().numpy()
    if not np.array_equal(a, rarg):
        i = tuple(np.argwhere(a != rarg)[0])
        raise AssertionError(f"{what}: argmax differs at {i}: gpu={a[i]} ref={rarg[i]}")


def run_propagate_case(pyg, ei_np, x_np, w_np=None, msg="src", aggr="sum", kernel="csr", dtype=torch.float32,
                       chunk=0, csr=None, what=""):
    """One propagate through the C ABI vs the oracle on identical inputs."""
    dev = torch.device("cuda")
    N = x_np.shape[0]
    x_in = x_np if dtype == torch.float32 else bf16_round(x_np)
    x = to_dev(x_np).to(dtype)
    ei = to_dev(ei_np)
    w = to_dev(w_np) if w_np is not None else None
    if kernel == "csr" and csr is None:
        csr = pyg.coo_to_csr(ei, N, w, chunk=chunk)
    out, arg = pyg.propagate(x, ei, w, csr=csr if kernel == "csr" else None, aggr=aggr, msg=msg, kernel=kernel)
    torch.cuda.synchronize(dev)
    ref, rarg, sabs = oracle.propagate(x_in, ei_np, w_np, msg=msg, aggr=aggr)
    tag = f"{what} {kernel} {msg} {aggr} {dtype} w={w_np is not None} chunk={chunk}"
    if aggr == "max":
        check_max(out, arg, ref, rarg, dtype == torch.bfloat16, tag)
        return 0.0
    return check_sum(out, ref, sabs, dtype == torch.bfloat16, tag)


def segment_max(s: np.ndarray, dst: np.ndarray, N: int) -> np.ndarray:
    """Per-target maximum of the scores [E, H] (used only for the tolerance)."""
    m = np.full((N, s.shape[1]), -np.inf)
    np.maximum.at(m, dst, s)
    return m


def check_softmax(gpu: torch.Tensor, ref: np.ndarray, s: np.ndarray, dst: np.ndarray, N: int, what: str = ""):
    g = gpu.float().cpu().numpy().astype(np.float64).reshape(ref.shape)
    s = np.asarray(s, np.float64).reshape(ref.shape)
    m = segment_max(s, dst, N)[dst] if s.size else s
    bound = ref * (1e-5 + 4 * 2.0**-24 * (np.abs(s) + np.abs(m) + 1)) + 1e-30
    err = np.abs(g - ref)
    bad = ~(err <= bound)
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: {bad.sum()} alphas out of tolerance; first {i} gpu={g[i]!r} ref={ref[i]!r} "
                             f"bound={bound[i]!r}")
    return float((err / bound).max()) if err.size else 0.0
