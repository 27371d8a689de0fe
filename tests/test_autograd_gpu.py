"""The autograd functions (GATAttention, PropagateEdge) inside torch
autograd: their gradients against the oracle's backward chains."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import check_sum, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


@pytest.mark.parametrize("N,E,H,C", [(50, 300, 2, 4), (2000, 30000, 8, 16), (700, 9000, 4, 3)])
def test_gat_attention_autograd(pyg, N, E, H, C):
    rng = np.random.default_rng(N + E)
    ei = synth.random_coo(rng, N, E)
    x = rng.standard_normal((N, H * C)).astype(np.float32)
    a_src = rng.standard_normal((N, H)).astype(np.float32)
    a_dst = rng.standard_normal((N, H)).astype(np.float32)
    g = rng.standard_normal((N, H * C)).astype(np.float32)
    graph = pyg.Graph(to_dev(ei), N)
    xt = to_dev(x).requires_grad_()
    st, dt = to_dev(a_src).requires_grad_(), to_dev(a_dst).requires_grad_()
    out = pyg.GATAttention.apply(xt, st, dt, graph, 0.2)
    out.backward(to_dev(g))
    torch.cuda.synchronize()
    e = oracle.gat_scores(a_src, a_dst, ei, 0.2)
    al = oracle.segment_softmax(e, ei, N)
    ref_out, sabs = oracle.propagate_heads(x, ei, al.astype(np.float32), H)
    assert np.all(np.abs(out.detach().cpu().numpy() - ref_out) <= 2e-5 * sabs + 1e-6), "forward"
    rx, ra, _, _ = oracle.propagate_heads_backward(x, ei, al.astype(np.float32), g, H)
    rsc, _ = oracle.segment_softmax_backward(al.astype(np.float32), ra.astype(np.float32), ei, N)
    rs, rd, _, _ = oracle.gat_scores_backward(a_src, a_dst, ei, rsc.astype(np.float32), 0.2)
    for got, ref, name in ((xt.grad, rx, "x"), (st.grad, rs, "a_src"), (dt.grad, rd, "a_dst")):
        err = np.abs(got.cpu().numpy().astype(np.float64) - ref).max()
        assert err <= 1e-4 * np.abs(ref).max() + 1e-6, f"grad {name}: {err}"


@pytest.mark.parametrize("msg", ["edge_add", "edge_relu", "edge_mul"])
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
def test_propagate_edge_autograd(pyg, msg, aggr):
    rng = np.random.default_rng(71)
    N, E, F = 800, 12000, 32
    ei = synth.random_coo(rng, N, E)
    x = rng.standard_normal((N, F)).astype(np.float32)
    ea = rng.standard_normal((E, F)).astype(np.float32)
    g = rng.standard_normal((N, F)).astype(np.float32)
    graph = pyg.Graph(to_dev(ei), N)
    xt, et = to_dev(x).requires_grad_(), to_dev(ea).requires_grad_()
    out = pyg.PropagateEdge.apply(xt, et, graph, msg, aggr)
    out.backward(to_dev(g))
    torch.cuda.synchronize()
    arg = None
    if aggr == "max":
        _, arg, _ = oracle.propagate(x, ei, msg=msg, aggr="max", edge_attr=ea)
    rx, re, sx, se = oracle.propagate_edge_backward(x, ei, ea, g, msg, aggr, argmax=arg)
    check_sum(xt.grad, rx, sx, False, f"PropagateEdge {msg} {aggr} grad_x")
    check_sum(et.grad, re, se, False, f"PropagateEdge {msg} {aggr} grad_e")


@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
def test_propagate_edge_autograd_bf16(pyg, aggr):
    """bf16 leaves: the gradients come back in bf16, against the oracle on
    the bf16-rounded values."""
    from tests.parity import bf16_round
    rng = np.random.default_rng(91)
    N, E, F = 600, 8000, 32
    ei = synth.random_coo(rng, N, E)
    x = bf16_round(rng.standard_normal((N, F)).astype(np.float32))
    ea = bf16_round(rng.standard_normal((E, F)).astype(np.float32))
    g = bf16_round(rng.standard_normal((N, F)).astype(np.float32))
    graph = pyg.Graph(to_dev(ei), N)
    for msg in ("edge_add", "edge_relu", "edge_mul"):
        xt = to_dev(x).bfloat16().requires_grad_()
        et = to_dev(ea).bfloat16().requires_grad_()
        out = pyg.PropagateEdge.apply(xt, et, graph, msg, aggr)
        assert out.dtype == torch.bfloat16
        out.backward(to_dev(g).bfloat16())
        torch.cuda.synchronize()
        assert xt.grad.dtype == torch.bfloat16 and et.grad.dtype == torch.bfloat16
        arg = None
        if aggr == "max":
            _, arg, _ = oracle.propagate(x, ei, msg=msg, aggr="max", edge_attr=ea)
        rx, re, sx, se = oracle.propagate_edge_backward(x, ei, ea, g, msg, aggr, argmax=arg)
        check_sum(xt.grad, rx, sx, True, f"PropagateEdge bf16 {msg} {aggr} grad_x")
        check_sum(et.grad, re, se, True, f"PropagateEdge bf16 {msg} {aggr} grad_e")


@pytest.mark.parametrize("aggr,msg", [("sum", "src"), ("mean", "src"), ("max", "src"), ("sum", "diff"),
                                      ("max", "diff")])
def test_propagate_autograd_unweighted_on_weighted_graph(pyg, aggr, msg):
    """A Graph built with weights, used without them: Eq. (1) with phi = x_j
    (or x_j - x_i) and its gradient, not the weighted propagate."""
    rng = np.random.default_rng(37)
    N, E, F = 600, 8000, 16
    ei = synth.random_coo(rng, N, E)
    x = rng.standard_normal((N, F)).astype(np.float32)
    w = rng.standard_normal(E).astype(np.float32)
    g = rng.standard_normal((N, F)).astype(np.float32)
    graph = pyg.Graph(to_dev(ei), N, to_dev(w))
    xt = to_dev(x).requires_grad_()
    out = pyg.Propagate.apply(xt, None, graph, aggr, msg)
    out.backward(to_dev(g))
    torch.cuda.synchronize()
    ref, rarg, sabs = oracle.propagate(x, ei, None, msg=msg, aggr=aggr)
    if aggr == "max":
        assert np.array_equal(out.detach().cpu().numpy(), ref.astype(np.float32)), "forward max"
    else:
        check_sum(out.detach(), ref, sabs, False, f"forward {aggr} {msg}")
    rx, _, sx, _ = oracle.propagate_backward(x, ei, g, None, msg=msg, aggr=aggr,
                                             argmax=rarg if aggr == "max" else None)
    check_sum(xt.grad, rx, sx, False, f"grad_x {aggr} {msg}")
