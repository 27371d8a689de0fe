"""Degenerate sizes on the backward and attention entry points: no nodes,
no edges, no feature columns. Every call must succeed and write zeros (or
nothing) without touching memory it was not given."""
import numpy as np
import pytest
import torch

import synth
from tests.parity import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def graphs(pyg, N, E):
    ei = synth.random_coo(np.random.default_rng(N + E), N, E) if N else np.zeros((2, 0), np.int64)
    d = to_dev(ei)
    csr = pyg.coo_to_csr(d, N)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(d), N)
    return d, csr, csr_t


@pytest.mark.parametrize("N,E", [(0, 0), (7, 0), (7, 30)])
def test_attention_backward_degenerate(pyg, N, E):
    d, csr, csr_t = graphs(pyg, N, E)
    H, C = 2, 4
    g = torch.randn(N, H * C, device="cuda")
    x = torch.randn(N, H * C, device="cuda")
    alpha = torch.rand(E, H, device="cuda")
    mt = pyg.csr_transpose_map(csr, csr_t)
    assert mt.shape == (E,)
    gx, ga = pyg.propagate_heads_backward(g, x, csr, csr_t, alpha, H, map_t=mt)
    a_s, a_d = torch.randn(N, H, device="cuda"), torch.randn(N, H, device="cuda")
    gs, gd = pyg.gat_scores_backward(a_s, a_d, csr, csr_t, torch.randn(E, H, device="cuda"), map_t=mt)
    torch.cuda.synchronize()
    assert gx.shape == (N, H * C) and ga.shape == (E, H) and gs.shape == (N, H) and gd.shape == (N, H)
    if E == 0:
        assert torch.count_nonzero(gx) == 0 and torch.count_nonzero(gs) == 0 and torch.count_nonzero(gd) == 0


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("N,E,F", [(0, 0, 4), (7, 0, 4), (7, 30, 0), (7, 30, 4)])
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
def test_edge_backward_degenerate(pyg, N, E, F, aggr, dtype):
    d, csr, csr_t = graphs(pyg, N, E)
    g = torch.randn(N, F, device="cuda").to(dtype)
    x = torch.randn(N, F, device="cuda").to(dtype)
    ea = torch.randn(E, F, device="cuda").to(dtype)
    arg = None
    if aggr == "max":
        _, arg = pyg.propagate_edge(x, ea, d, csr, "edge_relu", "max", "csr", "coo")
    gx, ge = pyg.propagate_edge_backward(g, x, ea, csr, "edge_relu", aggr, "coo", csr_t=csr_t, edge_index=d,
                                         argmax=arg)
    torch.cuda.synchronize()
    assert gx.shape == (N, F) and ge.shape == (E, F) and gx.dtype == dtype and ge.dtype == dtype
    if E == 0:
        assert torch.count_nonzero(gx) == 0


@pytest.mark.parametrize("N,E,F,D", [(0, 0, 4, 3), (7, 0, 4, 3), (7, 30, 0, 3), (7, 30, 4, 0), (7, 30, 4, 3)])
def test_edge_encoded_and_grad_w_order_degenerate(pyg, N, E, F, D):
    """The encoded edge propagate and grad_w in CSR order at empty sizes."""
    d, csr, csr_t = graphs(pyg, N, E)
    x = torch.randn(N, F, device="cuda")
    out, _ = pyg.propagate_edge_encoded(x, torch.randn(E, D, device="cuda"), torch.randn(D, F, device="cuda"), d, csr,
                                        "edge_relu", "sum", "csr", "coo")
    w = torch.rand(E, device="cuda")
    cw = pyg.coo_to_csr(d, N, w)
    cwt = pyg.coo_to_csr(pyg.reverse_edges(d), N, w)
    gx, gw = pyg.propagate_backward(torch.randn(N, F, device="cuda"), x, d, w, csr=cw, csr_t=cwt, aggr="sum",
                                    need_grad_w=True, w_order="csr")
    torch.cuda.synchronize()
    assert out.shape == (N, F) and gx.shape == (N, F) and gw.shape == (E,)
    if E == 0:
        assert torch.count_nonzero(out) == 0
    elif D == 0:  # no edge features: the message sees e = 0
        ref, _ = pyg.propagate_edge(x, torch.zeros(E, F, device="cuda"), d, csr, "edge_relu", "sum", "csr", "coo")
        assert torch.equal(out, ref)
    if F == 0:
        assert torch.count_nonzero(gw) == 0


def test_degree_csr_and_map_empty(pyg):
    d, csr, csr_t = graphs(pyg, 5, 0)
    assert torch.equal(pyg.degree_csr(csr).cpu(), torch.zeros(5, dtype=torch.int64))
    assert pyg.csr_transpose_map(csr, csr_t).numel() == 0


@pytest.mark.parametrize("N,E,F", [(0, 0, 4), (7, 0, 4), (7, 30, 0)])
def test_forward_calls_degenerate(pyg, N, E, F):
    d, csr, csr_t = graphs(pyg, N, E)
    x = torch.randn(N, F, device="cuda")
    for kernel in ("csr", "coo"):
        for aggr in ("sum", "mean", "max"):
            for dt in (torch.float32, torch.bfloat16):
                out, arg = pyg.propagate(x.to(dt), d, csr=csr if kernel == "csr" else None, aggr=aggr, kernel=kernel)
                assert out.shape == (N, F)
                if E == 0 and N * F:
                    assert torch.count_nonzero(out) == 0
                    if aggr == "max":
                        assert torch.all(arg == E)
    w = pyg.gcn_norm(d, N)
    assert w.shape == (E,)
    assert pyg.gcn_norm_csr(csr).shape == (E,)
    assert torch.equal(pyg.degree(d, N).cpu(), pyg.degree_csr(csr).cpu())
    H = 2
    s = torch.randn(E, H, device="cuda")
    assert pyg.segment_softmax(s, csr).shape == (E, H)
    assert pyg.gat_softmax(torch.randn(N, H, device="cuda"), torch.randn(N, H, device="cuda"), csr).shape == (E, H)
    assert pyg.segment_softmax_backward(s, s, csr).shape == (E, H)
    batch = torch.zeros(N, dtype=torch.int64, device="cuda")
    for aggr in ("sum", "mean", "max"):
        pooled, _ = pyg.global_pool(x, batch, 1, aggr)
        assert pooled.shape == (1, F)
        if N == 0 and F:
            assert torch.count_nonzero(pooled) == 0
    if F % 8 == 0:
        t = torch.randn(F, 16, device="cuda").to(torch.bfloat16)
        assert pyg.dense_transform(x.to(torch.bfloat16), t).shape == (N, 16)
        assert pyg.dense_transform(x.float(), t.float()).shape == (N, 16)
    torch.cuda.synchronize()
