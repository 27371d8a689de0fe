"""The allocation-free propagate (pyg_propagate_noalloc, scratch in a static
per-GPU device array) against pyg_propagate (caller workspace) on the same
inputs, through the C ABI: two calls in a row, the second on a smaller graph,
so that the second call runs on scratch the first one left behind.

CSR results are deterministic, so they must agree bit for bit; the COO
kernel's float atomics make sum / mean order-dependent, so those are held to
the parity rule against the oracle (|a - ref| <= 1e-5 * S + 1e-6 on both
sides), max / argmax bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import check_max, check_sum, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    m.library()
    return m


def _inputs(cfg):
    c = synth.make_config(cfg, seed=0)
    ei_np, x_np, N = c["edge_index_gcn"], c["x"], c["N"]
    w_np = oracle.gcn_norm(ei_np, N).astype(np.float32)
    return ei_np, x_np, w_np, N


def _same(a: torch.Tensor, b: torch.Tensor, what: str):
    if a.dtype == torch.float32:
        ok = torch.equal(a.view(torch.int32), b.view(torch.int32))
    else:
        ok = torch.equal(a, b)
    assert ok, f"{what}: noalloc result differs from pyg_propagate"


@pytest.mark.parametrize("kernel", ["csr", "coo"])
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_noalloc_matches_workspace_call(pyg, kernel, aggr, dtype):
    # the PubMed-shaped graph (F = 64, hub rows folded across chunks), then
    # the smaller Cora-shaped one (F = 16)
    for cfg in (2, 1):
        ei_np, x_np, w_np, N = _inputs(cfg)
        xin = x_np if dtype == torch.float32 else x_np.astype(np.float32)
        x = to_dev(xin).to(dtype)
        ei = to_dev(ei_np)
        w = to_dev(w_np)
        csr = pyg.coo_to_csr(ei, N, w) if kernel == "csr" else None
        out_ref, arg_ref = pyg.propagate(x, ei, w, csr=csr, aggr=aggr, kernel=kernel)
        out = torch.full_like(x, float("nan"))
        arg = torch.full((N, x.shape[1]), -7, dtype=torch.int64, device=x.device) if aggr == "max" else None
        out2, arg2 = pyg.propagate_noalloc(x, ei, w, csr=csr, aggr=aggr, kernel=kernel, out=out, argmax=arg)
        torch.cuda.synchronize()
        assert out2.data_ptr() == out.data_ptr()
        tag = f"config {cfg} {kernel} {aggr} {dtype}"
        if kernel == "csr" or aggr == "max":
            _same(out, out_ref, tag)
            if aggr == "max":
                assert torch.equal(arg2, arg_ref), f"{tag}: argmax differs"
            continue
        x_or = x.float().cpu().numpy()
        ref, rarg, sabs = oracle.propagate(x_or, ei_np, w_np, aggr=aggr)
        bf = dtype == torch.bfloat16
        check_sum(out, ref, sabs, bf, tag + " noalloc")
        check_sum(out_ref, ref, sabs, bf, tag + " workspace")


def test_noalloc_max_against_oracle(pyg):
    # the second, smaller call checked against the oracle too (not only
    # against the workspace entry point)
    for cfg in (2, 1):
        ei_np, x_np, w_np, N = _inputs(cfg)
        ei, x, w = to_dev(ei_np), to_dev(x_np), to_dev(w_np)
        csr = pyg.coo_to_csr(ei, N, w)
        out, arg = pyg.propagate_noalloc(x, ei, w, csr=csr, aggr="max")
        torch.cuda.synchronize()
        ref, rarg, _ = oracle.propagate(x_np, ei_np, w_np, aggr="max")
        check_max(out, arg, ref, rarg, False, f"config {cfg} noalloc max")


def test_noalloc_rejects_oversized_call(pyg):
    # max over the COO kernel keeps N*F 8-byte keys in scratch: 2^20 x 128
    # needs 1 GiB, beyond the static array; rejected before any device work
    N, F = 1 << 20, 128
    x = torch.empty((N, F), dtype=torch.float32, device="cuda")
    ei = torch.zeros((2, 4), dtype=torch.int64, device="cuda")
    with pytest.raises(pyg.PygError) as e:
        pyg.propagate_noalloc(x, ei, aggr="max", kernel="coo")
    assert e.value.status == -5
