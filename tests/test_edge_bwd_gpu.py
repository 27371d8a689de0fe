"""GPU parity of the edge-feature message gradients (pyg_propagate_edge_backward)
against the oracle: every message, aggregation and feature order, on small
random multigraphs, a graph with a hub row over many chunks and a
power-law-like spread of row lengths. The max path takes the oracle's
forward argmax as its input on both sides."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_sum, to_dev

pytestmark = pytest.mark.gpu

MSGS = ["edge_add", "edge_relu", "edge_mul"]


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def case(pyg, ei, N, F, seed, msg, aggr, order, chunk=0, use_map=False, dtype=torch.float32):
    rng = np.random.default_rng(seed)
    E = ei.shape[1]
    x = rng.standard_normal((N, F)).astype(np.float32)
    ea = rng.standard_normal((E, F)).astype(np.float32)
    g = rng.standard_normal((N, F)).astype(np.float32)
    bf16 = dtype == torch.bfloat16
    if bf16:  # the oracle sees exactly the values the device holds
        x, ea, g = bf16_round(x), bf16_round(ea), bf16_round(g)
    d_ei = to_dev(ei)
    csr = pyg.coo_to_csr(d_ei, N, chunk=chunk)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N, chunk=chunk)
    _, _, perm = oracle.coo_to_csr(ei, N)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)
    arg = None
    if aggr == "max":
        _, arg, _ = oracle.propagate(x, ei, msg=msg, aggr="max", edge_attr=ea)
    rx, re, sx, se = oracle.propagate_edge_backward(x, ei, ea, g, msg, aggr, argmax=arg)
    ea_in = ea[perm] if order == "csr" else ea
    mt = pyg.csr_transpose_map(csr, csr_t) if use_map else None
    gx, ge = pyg.propagate_edge_backward(to_dev(g).to(dtype), to_dev(x).to(dtype), to_dev(ea_in).to(dtype), csr, msg,
                                         aggr, order, csr_t=csr_t, map_t=mt, edge_index=d_ei,
                                         argmax=None if arg is None else to_dev(arg))
    torch.cuda.synchronize()
    assert gx.dtype == dtype and ge.dtype == dtype
    tag = f"edge bwd {msg} {aggr} {order} {dtype} N={N} E={E} F={F} chunk={chunk}"
    check_sum(gx, rx, sx, bf16, tag + " grad_x")
    ge_coo = ge.float().cpu().numpy()
    if order == "csr" and E:
        back = np.empty_like(ge_coo)
        back[perm] = ge_coo
        ge_coo = back
    check_sum(torch.from_numpy(ge_coo), re, se, bf16, tag + " grad_e")


GRAPHS = [(1, 0, 3), (5, 1, 4), (60, 400, 1), (300, 5000, 7), (2000, 30000, 16), (700, 9000, 128), (257, 4000, 130)]


@pytest.mark.parametrize("order", ["csr", "coo"])
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
def test_edge_backward(pyg, aggr, order):
    for i, (N, E, F) in enumerate(GRAPHS):
        ei = synth.random_coo(np.random.default_rng(40 + i), N, E)
        for j, msg in enumerate(MSGS):
            case(pyg, ei, N, F, 500 + 10 * i + j, msg, aggr, order, use_map=(i + j) % 2 == 1)


@pytest.mark.parametrize("chunk", [0, 64])
def test_edge_backward_hub_and_graded_rows(pyg, chunk):
    rng = np.random.default_rng(61)
    ei = synth.random_coo(rng, 3000, 40000)
    ei[1, :20000] = 0  # one hub row across many chunks
    for msg in MSGS:
        for aggr in ("sum", "mean", "max"):
            case(pyg, ei, 3000, 32, 62, msg, aggr, "csr", chunk=chunk)
    deg = np.unique(np.geomspace(1, 3000, 80).astype(np.int64))
    ei = synth.graded_in_degree(rng, 200, deg)
    for msg in MSGS:
        case(pyg, ei, 200, 64, 63, msg, "sum", "coo", chunk=chunk, use_map=True)


def test_edge_backward_outputs_optional_and_deterministic(pyg):
    rng = np.random.default_rng(64)
    N, E, F = 3000, 60000, 32
    ei = synth.random_coo(rng, N, E)
    d_ei = to_dev(ei)
    csr = pyg.coo_to_csr(d_ei, N, chunk=64)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N, chunk=64)
    x, ea, g = torch.randn(N, F, device="cuda"), torch.randn(E, F, device="cuda"), torch.randn(N, F, device="cuda")
    for msg in MSGS:
        gx, ge = pyg.propagate_edge_backward(g, x, ea, csr, msg, "sum", "csr", csr_t=csr_t)
        gx2, none = pyg.propagate_edge_backward(g, x, ea, csr, msg, "sum", "csr", csr_t=csr_t, need_grad_edge=False)
        none2, ge2 = pyg.propagate_edge_backward(g, x, ea, csr, msg, "sum", "csr", need_grad_x=False)
        assert none is None and none2 is None
        assert torch.equal(gx, gx2) and torch.equal(ge, ge2)


def test_edge_backward_bf16(pyg):
    """bf16 operands and gradients: every message, aggregation and order,
    against the oracle on the bf16-rounded inputs (one rounding of each
    gradient allowed on top of the fp32 bound)."""
    for i, (N, E, F) in enumerate(GRAPHS):
        ei = synth.random_coo(np.random.default_rng(70 + i), N, E)
        for j, msg in enumerate(MSGS):
            for k, aggr in enumerate(("sum", "mean", "max")):
                order = "csr" if (i + j + k) % 2 == 0 else "coo"
                case(pyg, ei, N, F, 700 + 10 * i + j, msg, aggr, order, use_map=(i + k) % 2 == 1,
                     dtype=torch.bfloat16)


@pytest.mark.parametrize("chunk", [0, 64])
def test_edge_backward_bf16_hub(pyg, chunk):
    rng = np.random.default_rng(66)
    ei = synth.random_coo(rng, 3000, 40000)
    ei[1, :20000] = 0
    for msg in MSGS:
        for aggr in ("sum", "mean", "max"):
            case(pyg, ei, 3000, 32, 67, msg, aggr, "csr", chunk=chunk, dtype=torch.bfloat16)


def test_edge_backward_bf16_matches_f32_rounded(pyg):
    """Under sum each edge gradient is one fp32 product or gate of the same
    widened bf16 values in both paths, so bf16 grad_e is the fp32 path's
    rounded once, bit for bit; grad_x sums in fp32 in a lane layout of its
    own, so it may differ by the bf16 rounding of last-bit fp32 differences."""
    rng = np.random.default_rng(68)
    N, E, F = 2000, 30000, 64
    d_ei = to_dev(synth.random_coo(rng, N, E))
    csr = pyg.coo_to_csr(d_ei, N)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N)
    x = torch.randn(N, F, device="cuda").bfloat16()
    ea = torch.randn(E, F, device="cuda").bfloat16()
    g = torch.randn(N, F, device="cuda").bfloat16()
    for msg in MSGS:
        gx, ge = pyg.propagate_edge_backward(g, x, ea, csr, msg, "sum", "csr", csr_t=csr_t)
        fx, fe = pyg.propagate_edge_backward(g.float(), x.float(), ea.float(), csr, msg, "sum", "csr", csr_t=csr_t)
        assert torch.equal(ge.view(torch.int16), fe.bfloat16().view(torch.int16)), msg
        assert torch.allclose(gx.float(), fx, rtol=2.0 ** -8, atol=1e-4), msg
