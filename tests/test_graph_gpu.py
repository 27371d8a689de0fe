"""The whole step (coo_to_csr -> degree_csr -> gcn_norm_csr -> propagate ->
global mean pool) captured once in a HIP graph and replayed. The library
allocates nothing, never synchronises with the host and clears memory with
kernels (no memset nodes), so every call can be captured. Each replay, with
eager runs of the same step in between, must reproduce the eager outputs
bit for bit: every kernel of the step has a fixed reduction order."""
import ctypes

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


def make_step(pyg, ei_np, N, x_np, batch_np, B):
    """All outputs and workspaces preallocated; returns (step, outputs)."""
    dev = torch.device("cuda")
    lib = pyg.library()
    E = ei_np.shape[1]
    ei, x, batch = to_dev(ei_np), to_dev(x_np), to_dev(batch_np)
    F = x.shape[1]
    csr = pyg.CSR(torch.empty(N + 1, dtype=torch.int64, device=dev), torch.empty(E, dtype=torch.int32, device=dev),
                  torch.empty(E, dtype=torch.int64, device=dev), None, N, E, 0)
    norm = torch.empty(E, dtype=torch.float32, device=dev)
    csr_w = pyg.CSR(csr.rowptr, csr.col, csr.perm, norm, N, E, 0)
    deg = torch.empty(N, dtype=torch.int64, device=dev)
    out = torch.empty_like(x)
    pooled = torch.empty(B, F, dtype=torch.float32, device=dev)
    sz = ctypes.c_size_t()

    def ws(fn, *a):
        assert fn(*a, ctypes.byref(sz)) == 0
        return torch.empty(max(sz.value, 1), dtype=torch.uint8, device=dev)
    ws_csr = ws(lib.pyg_coo_to_csr_workspace, E, N)
    ws_norm = ws(lib.pyg_gcn_norm_csr_workspace, N)
    ws_pool = ws(lib.pyg_global_pool_workspace, 0, N, F, B, 1)
    ws_prop = torch.empty(pyg.propagate_workspace_bytes(x, E, "sum", "csr", 0), dtype=torch.uint8, device=dev)

    def step():
        pyg.coo_to_csr(ei, N, None, out=csr, workspace=ws_csr)
        pyg.degree_csr(csr, out=deg)
        pyg.gcn_norm_csr(csr, out=norm, workspace=ws_norm)
        pyg.propagate(x, csr=csr_w, aggr="sum", out=out, workspace=ws_prop)
        pyg.global_pool(out, batch, B, "mean", out=pooled, workspace=ws_pool)

    return step, {"rowptr": csr.rowptr, "col": csr.col, "perm": csr.perm, "deg": deg, "norm": norm, "out": out,
                  "pooled": pooled}


def graphs():
    c1 = synth.make_config(1)
    yield "cora-shaped", c1["edge_index_gcn"], c1["N"], c1["x"], np.zeros(c1["N"], np.int64), 1
    c3 = synth.make_config(3)
    yield "mini-batch", c3["edge_index"], c3["N"], c3["x"], c3["batch"], c3["B"]
    rng = np.random.default_rng(5)
    N = 20000
    ei = synth.with_self_loops(synth.random_coo(rng, N, 300000), N)
    yield "random 20k", ei, N, rng.standard_normal((N, 64)).astype(np.float32), np.sort(rng.integers(0, 7, N)), 7


@pytest.mark.parametrize("which", [0, 1, 2])
def test_step_graph_replay(pyg, which):
    name, ei, N, x, batch, B = list(graphs())[which]
    step, outs = make_step(pyg, ei, N, x, batch, B)
    # warm up on a side stream (default priority), as capture requires
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    step()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in outs.items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        for v in outs.values():  # scribble over every output, eagerly
            v.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v, ref[k]), f"{name}: replay {r} differs in {k}"
        step()  # the program's own eager work between replays
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v, ref[k]), f"{name}: eager run after replay {r} differs in {k}"


def test_training_sequence_graph_replay(pyg):
    """A training-shaped sequence captured as it is called from Python (the
    binding's own output and workspace allocations come from the graph's
    memory pool): weighted propagate, its backward with grad_w in both
    orders, GAT coefficients and the attention sum. Every replay must equal
    the eager results bit for bit."""
    rng = np.random.default_rng(77)
    N, E, F, H = 3000, 40000, 64, 4
    ei = to_dev(synth.random_coo(rng, N, E))
    w = torch.rand(E, device="cuda")
    x = torch.randn(N, F, device="cuda")
    g = torch.randn(N, F, device="cuda")
    a_s, a_d = torch.randn(N, H, device="cuda"), torch.randn(N, H, device="cuda")
    csr = pyg.coo_to_csr(ei, N, w)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, w)
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, E, csr.chunk)

    def seq():
        out, _ = pyg.propagate(x, csr=csr, aggr="sum")
        gx, gw = pyg.propagate_backward(g, x, ei, w, csr=csr, csr_t=csr_t, aggr="sum", need_grad_w=True)
        _, gwc = pyg.propagate_backward(g, x, ei, w, csr=csr, csr_t=csr_t, aggr="sum", need_grad_w=True,
                                        w_order="csr")
        alpha = pyg.gat_softmax(a_s, a_d, plain, order="csr")
        att = pyg.propagate_heads(x, plain, alpha, H)
        return [out, gx, gw, gwc, alpha, att]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        seq()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref = [t.clone() for t in seq()]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        outs = seq()
    torch.cuda.synchronize()
    for r in range(3):
        for t in outs:
            t.fill_(-1)
        graph.replay()
        torch.cuda.synchronize()
        for i, (t, rr) in enumerate(zip(outs, ref)):
            assert torch.equal(t, rr), f"replay {r}: output {i} differs"
        again = seq()  # eager work between replays
        torch.cuda.synchronize()
        for i, (t, rr) in enumerate(zip(again, ref)):
            assert torch.equal(t, rr), f"eager after replay {r}: output {i} differs"
