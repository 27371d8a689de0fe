"""GPU parity of pyg_propagate_backward against the oracle's backward on
identical seeded inputs (max: both sides take the oracle's forward argmax)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_sum, to_dev

pytestmark = pytest.mark.gpu

F32, BF16 = torch.float32, torch.bfloat16

# (N, E, F): chunk-spanning sizes, ragged tails, light and heavy rows, odd F
CASES = [(1, 4, 3), (9, 0, 8), (60, 400, 1), (300, 5000, 16), (2000, 30000, 64), (700, 9000, 128),
         (400, 3000, 500), (257, 4000, 260)]


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def run_case(pyg, N, E, F, seed, aggr, msg, dtype, chunk=0, hub=False):
    rng = np.random.default_rng(seed)
    ei = synth.random_coo(rng, N, E)
    if hub and E:  # a mega-hub target and source: long rows in both directions
        ei[1, : E // 2] = 0
        ei[0, E // 2:] = 1
    x = rng.standard_normal((N, F)).astype(np.float32)
    g = rng.standard_normal((N, F)).astype(np.float32)
    w = rng.standard_normal(E).astype(np.float32) if msg == "weighted" else None
    m = "diff" if msg == "diff" else "src"
    if dtype == BF16:
        x, g = bf16_round(x), bf16_round(g)
    argmax = None
    if aggr == "max":
        _, argmax, _ = oracle.propagate(x, ei, w, msg=m, aggr="max")
    ref_x, ref_w, sx, sw = oracle.propagate_backward(x, ei, g, w, msg=m, aggr=aggr, argmax=argmax,
                                                     want_grad_w=w is not None)
    d_ei = to_dev(ei)
    d_w = to_dev(w) if w is not None else None
    csr = csr_t = None
    if aggr != "max":
        csr = pyg.coo_to_csr(d_ei, N, d_w, chunk=chunk)
        csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N, d_w, chunk=chunk)
    gx, gw = pyg.propagate_backward(to_dev(g).to(dtype), to_dev(x).to(dtype), d_ei, d_w, csr, csr_t, aggr, m,
                                    to_dev(argmax) if argmax is not None else None, need_grad_w=w is not None)
    torch.cuda.synchronize()
    tag = f"bwd N={N} E={E} F={F} {aggr} {msg} {dtype} chunk={chunk}"
    check_sum(gx, ref_x, sx, dtype == BF16, tag + " grad_x")
    if w is not None:
        check_sum(gw, ref_w, sw, False, tag + " grad_w")


COMBOS = [(a, m, d) for a in ("sum", "mean", "max") for m in ("src", "weighted", "diff") for d in (F32, BF16)]


@pytest.mark.parametrize("aggr,msg,dtype", COMBOS, ids=[f"{a}-{m}-{str(d)[6:]}" for a, m, d in COMBOS])
def test_backward_small(pyg, aggr, msg, dtype):
    for i, (N, E, F) in enumerate(CASES):
        run_case(pyg, N, E, F, 100 + i, aggr, msg, dtype)


@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
@pytest.mark.parametrize("chunk", [0, 64])
def test_backward_hubs(pyg, aggr, chunk):
    for msg in ("src", "weighted", "diff"):
        run_case(pyg, 3000, 20000, 32, 7, aggr, msg, F32, chunk=chunk, hub=True)


def test_backward_sum_is_deterministic(pyg):
    rng = np.random.default_rng(3)
    N, E, F = 5000, 80000, 64
    ei = to_dev(synth.random_coo(rng, N, E))
    g = torch.randn(N, F, device="cuda")
    x = torch.randn(N, F, device="cuda")
    w = torch.randn(E, device="cuda")
    csr = pyg.coo_to_csr(ei, N, w)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, w)
    first = pyg.propagate_backward(g, x, ei, w, csr, csr_t, "mean", need_grad_w=True)
    for _ in range(3):
        again = pyg.propagate_backward(g, x, ei, w, csr, csr_t, "mean", need_grad_w=True)
        assert torch.equal(again[0], first[0]) and torch.equal(again[1], first[1])


def test_backward_config2(pyg):
    """The power-law workload with its gcn_norm weights, F = 64."""
    c = synth.make_config(2, F=64)
    N, ei = c["N"], c["edge_index_gcn"]
    w = oracle.gcn_norm(ei, N).astype(np.float32)
    x = c["x"]
    g = np.random.default_rng(5).standard_normal(x.shape).astype(np.float32)
    d_ei, d_w = to_dev(ei), to_dev(w)
    csr = pyg.coo_to_csr(d_ei, N, d_w)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N, d_w)
    for aggr in ("sum", "mean"):
        gx, gw = pyg.propagate_backward(to_dev(g), to_dev(x), d_ei, d_w, csr, csr_t, aggr, need_grad_w=True)
        rx, rw, sx, sw = oracle.propagate_backward(x, ei, g, w, aggr=aggr, want_grad_w=True)
        check_sum(gx, rx, sx, what=f"C2 bwd {aggr} grad_x")
        check_sum(gw, rw, sw, what=f"C2 bwd {aggr} grad_w")
    _, argmax, _ = oracle.propagate(x, ei, w, aggr="max")
    gx, gw = pyg.propagate_backward(to_dev(g), to_dev(x), d_ei, d_w, aggr="max", argmax=to_dev(argmax), need_grad_w=True)
    rx, rw, sx, sw = oracle.propagate_backward(x, ei, g, w, aggr="max", argmax=argmax, want_grad_w=True)
    check_sum(gx, rx, sx, what="C2 bwd max grad_x")
    check_sum(gw, rw, sw, what="C2 bwd max grad_w")


def test_autograd_function(pyg):
    """Propagate.apply inside torch autograd gives the oracle's gradients."""
    rng = np.random.default_rng(12)
    N, E, F = 800, 9000, 32
    ei = synth.random_coo(rng, N, E)
    x = rng.standard_normal((N, F)).astype(np.float32)
    w = rng.standard_normal(E).astype(np.float32)
    g = rng.standard_normal((N, F)).astype(np.float32)
    graph = pyg.Graph(to_dev(ei), N, to_dev(w))
    for aggr in ("sum", "mean", "max"):
        xt = to_dev(x).requires_grad_(True)
        wt = to_dev(w).requires_grad_(True)
        out = pyg.Propagate.apply(xt, wt, graph, aggr, "src")
        out.backward(to_dev(g))
        ref, arg, s = oracle.propagate(x, ei, w, aggr=aggr)
        check_sum(out.detach(), ref, s, what=f"autograd fwd {aggr}")
        rx, rw, sx, sw = oracle.propagate_backward(x, ei, g, w, aggr=aggr, argmax=arg, want_grad_w=True)
        check_sum(xt.grad, rx, sx, what=f"autograd grad_x {aggr}")
        check_sum(wt.grad, rw, sw, what=f"autograd grad_w {aggr}")


@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32", "bf16"])
def test_backward_grad_w_csr_order(pyg, aggr, dtype):
    """grad_w in CSR slot order: under sum / mean the same dot products as the
    COO order, stored at the slot instead of the edge id (bit for bit); under
    max the atomically summed entries against the oracle, re-ordered by the
    CSR permutation."""
    for i, (N, E, F) in enumerate([(300, 5000, 16), (2000, 30000, 64), (700, 9000, 128), (257, 4000, 260)]):
        rng = np.random.default_rng(300 + i)
        ei = synth.random_coo(rng, N, E)
        x = rng.standard_normal((N, F)).astype(np.float32)
        g = rng.standard_normal((N, F)).astype(np.float32)
        w = rng.standard_normal(E).astype(np.float32)
        if dtype == BF16:
            x, g = bf16_round(x), bf16_round(g)
        d_ei, d_w = to_dev(ei), to_dev(w)
        csr = pyg.coo_to_csr(d_ei, N, d_w)
        csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N, d_w)
        _, _, perm = oracle.coo_to_csr(ei, N)
        argmax = None
        if aggr == "max":
            _, argmax, _ = oracle.propagate(x, ei, w, aggr="max")
        args = dict(argmax=to_dev(argmax) if argmax is not None else None, need_grad_w=True)
        gd, xd = to_dev(g).to(dtype), to_dev(x).to(dtype)
        gx_coo, gw_coo = pyg.propagate_backward(gd, xd, d_ei, d_w, csr, csr_t, aggr, **args)
        gx_csr, gw_csr = pyg.propagate_backward(gd, xd, d_ei, d_w, csr, csr_t, aggr, w_order="csr", **args)
        torch.cuda.synchronize()
        tag = f"grad_w csr order N={N} E={E} F={F} {aggr} {dtype}"
        if aggr != "max":
            assert torch.equal(gx_csr, gx_coo), tag
            assert torch.equal(gw_csr, gw_coo[torch.from_numpy(perm).cuda()]), tag
        _, ref_w, _, sw = oracle.propagate_backward(x, ei, g, w, aggr=aggr, argmax=argmax, want_grad_w=True)
        check_sum(gw_csr, ref_w[perm], sw[perm], False, tag)
