"""GPU parity of the matrix-core dense transform X Theta (bf16 operands,
fp32 accumulation) against the fp64 oracle on the same bf16 values, and of
a GCN layer (transform, then gcn_norm-weighted propagate) against the
oracle chain."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_sum, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


# (N, Fi, Fo): ragged rows and columns, Fi not a multiple of 8 (scalar path),
# several 128-column passes, K above one 128 chunk (PubMed's 500, Reddit's 602)
SHAPES = [(1, 1, 1), (5, 8, 16), (100, 16, 7), (1000, 128, 128), (333, 500, 64), (257, 40, 300), (70, 13, 5),
          (0, 8, 8), (4097, 602, 41), (129, 32, 129)]


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_dense_transform(pyg, out_dtype):
    for i, (N, Fi, Fo) in enumerate(SHAPES):
        rng = np.random.default_rng(600 + i)
        x = bf16_round(rng.standard_normal((N, Fi)).astype(np.float32))
        t = bf16_round((rng.standard_normal((Fi, Fo)) / np.sqrt(max(Fi, 1))).astype(np.float32))
        got = pyg.dense_transform(to_dev(x).to(torch.bfloat16), to_dev(t).to(torch.bfloat16), out_dtype)
        torch.cuda.synchronize()
        ref, sabs = oracle.dense_transform(x, t)
        check_sum(got, ref, sabs, out_dtype == torch.bfloat16, f"dense N={N} Fi={Fi} Fo={Fo} {out_dtype}")


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_dense_transform_f32_operands(pyg, out_dtype):
    """fp32 X and Theta on the fp32 matrix-core path, against the fp64 oracle
    on the same fp32 values (ragged shapes, Fi not a multiple of 4, several K
    chunks of 64 and column passes of 128)."""
    for i, (N, Fi, Fo) in enumerate(SHAPES + [(500, 66, 130), (64, 3, 200)]):
        rng = np.random.default_rng(650 + i)
        x = rng.standard_normal((N, Fi)).astype(np.float32)
        t = (rng.standard_normal((Fi, Fo)) / np.sqrt(max(Fi, 1))).astype(np.float32)
        got = pyg.dense_transform(to_dev(x), to_dev(t), out_dtype)
        torch.cuda.synchronize()
        assert got.dtype == out_dtype
        ref, sabs = oracle.dense_transform(x, t)
        check_sum(got, ref, sabs, out_dtype == torch.bfloat16, f"dense f32 N={N} Fi={Fi} Fo={Fo} {out_dtype}")


def test_dense_transform_f32_unaligned_and_deterministic(pyg):
    """An fp32 view whose rows start 4 bytes off a 16-byte boundary takes the
    scalar loads; repeated calls give identical bits."""
    rng = np.random.default_rng(19)
    base_np = rng.standard_normal(301 * 64 + 1).astype(np.float32)
    t_np = (rng.standard_normal((64, 48)) / 8).astype(np.float32)
    base, t = to_dev(base_np), to_dev(t_np)
    xo = base[1:].view(301, 64)
    got = pyg.dense_transform(xo, t)
    torch.cuda.synchronize()
    ref, sabs = oracle.dense_transform(base_np[1:].reshape(301, 64), t_np)
    check_sum(got, ref, sabs, False, "dense f32 unaligned")
    x = torch.randn(5000, 128, device="cuda")
    tt = torch.randn(128, 96, device="cuda") / 11
    first = pyg.dense_transform(x, tt)
    for _ in range(3):
        assert torch.equal(pyg.dense_transform(x, tt), first)
    with pytest.raises(ValueError):
        pyg.dense_transform(x, tt.to(torch.bfloat16))  # operands of two types


def test_dense_transform_unaligned_rows(pyg):
    """A view whose rows start off a 16-byte boundary takes the scalar path."""
    rng = np.random.default_rng(9)
    base_np = bf16_round(rng.standard_normal((301, 65)).astype(np.float32))
    t_np = bf16_round(rng.standard_normal((64, 32)).astype(np.float32) / 8)
    base = to_dev(base_np).to(torch.bfloat16)
    x = base[:, 1:].contiguous()[:, :64]  # contiguous copy, aligned
    xo = base.view(-1)[1:1 + 300 * 64].view(300, 64)  # offset by 2 bytes
    t = to_dev(t_np).to(torch.bfloat16)
    # the same values on the host, for the oracle
    x_np = np.ascontiguousarray(base_np[:300, 1:65])
    xo_np = base_np.reshape(-1)[1:1 + 300 * 64].reshape(300, 64)
    for xx, xh in ((x[:300], x_np), (xo, xo_np)):
        got = pyg.dense_transform(xx, t)
        torch.cuda.synchronize()
        ref, sabs = oracle.dense_transform(xh, t_np)
        check_sum(got, ref, sabs, False, "dense unaligned")


def test_dense_transform_deterministic(pyg):
    x = torch.randn(5000, 128, device="cuda").to(torch.bfloat16)
    t = (torch.randn(128, 96, device="cuda") / 11).to(torch.bfloat16)
    first = pyg.dense_transform(x, t)
    for _ in range(3):
        assert torch.equal(pyg.dense_transform(x, t), first)


def test_gcn_layer_chain(pyg):
    """A GCN layer on the PubMed-shaped graph: X Theta (500 -> 64) on the
    matrix cores, then the gcn_norm-weighted CSR propagate, against the
    oracle chain.
    fp32 intermediate: both stages are sums, so the error stays within
    1e-5 S + 1e-6 with S = sum_k |w_k| S_h[j_k] + sum_k |w_k h_j| (S_h the
    transform's sum of |terms|).
    bf16 intermediate: the GPU rounds its fp32 X Theta and the oracle its fp64
    one; the two bf16 values differ by at most one bf16 ulp (2^-7 relative),
    so the output may move by 2^-7 sum |w h| beyond the bf16 rule."""
    c = synth.make_config(2, F=500)
    N, ei = c["N"], c["edge_index_gcn"]
    rng = np.random.default_rng(10)
    x = bf16_round(c["x500"])
    t = bf16_round((rng.standard_normal((500, 64)) / np.sqrt(500)).astype(np.float32))
    w = oracle.gcn_norm(ei, N).astype(np.float32)
    d_ei, d_w = to_dev(ei), to_dev(w)
    csr = pyg.coo_to_csr(d_ei, N, d_w)
    xb, tb = to_dev(x).to(torch.bfloat16), to_dev(t).to(torch.bfloat16)
    href, hsabs = oracle.dense_transform(x, t)
    # fp32 intermediate
    h = pyg.dense_transform(xb, tb, torch.float32)
    out, _ = pyg.propagate(h, d_ei, d_w, csr=csr, aggr="sum")
    torch.cuda.synchronize()
    ref, _, sabs = oracle.propagate(href.astype(np.float32), ei, w, aggr="sum")
    carried, _, _ = oracle.propagate(hsabs.astype(np.float32), ei, np.abs(w), aggr="sum")
    check_sum(out, ref, sabs + carried, False, "gcn layer chain (fp32 intermediate)")
    # bf16 intermediate
    hb = pyg.dense_transform(xb, tb, torch.bfloat16)
    outb, _ = pyg.propagate(hb, d_ei, d_w, csr=csr, aggr="sum")
    torch.cuda.synchronize()
    refb, _, sabsb = oracle.propagate(bf16_round(href.astype(np.float32)), ei, w, aggr="sum")
    g = outb.float().cpu().numpy().astype(np.float64)
    bound = 1e-2 * np.abs(refb) + (2.0 ** -7 + 1e-5) * sabsb + 1e-6
    assert np.all(np.abs(g - refb) <= bound), f"gcn layer chain (bf16): worst {np.max(np.abs(g - refb) / bound)}"
