"""Graphs whose rows have long runs without edges (leading, interior and
trailing runs of target ids with no incoming edge, as when a bipartite graph
is padded into one node range): every walker over CSR rows must give the
oracle's result there (zeros for the empty rows, argmax = sentinel) and skip
the runs rather than step through them."""
import numpy as np
import pytest
import torch

import oracle
from tests.parity import check_max, check_softmax, check_sum, to_dev

pytestmark = pytest.mark.gpu

F32 = torch.float32


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def runs_graph(rng, N, E):
    """Targets only in [N/5, 2N/5) and [3N/5, 4N/5): runs of N/5 empty rows at
    the start, in the middle and at the end; sources anywhere."""
    q = N // 5
    dst = np.where(rng.random(E) < 0.5, rng.integers(q, 2 * q, E), rng.integers(3 * q, 4 * q, E))
    src = rng.integers(0, N, E)
    return np.stack([src, dst]).astype(np.int64)


# (N, E): light rows (mean degree over the non-empty rows 15) and heavy ones (100)
GRAPHS = [(20000, 120000), (20000, 800000)]


@pytest.mark.parametrize("N,E", GRAPHS)
@pytest.mark.parametrize("F", [16, 128])
def test_propagate_empty_runs(pyg, N, E, F):
    rng = np.random.default_rng(N + E + F)
    ei_np = runs_graph(rng, N, E)
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    w_np = rng.standard_normal(E).astype(np.float32)
    ei, x = to_dev(ei_np), to_dev(x_np)
    csr = pyg.coo_to_csr(ei, N, to_dev(w_np))
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, E, csr.chunk)
    for aggr in ("sum", "mean"):
        out, _ = pyg.propagate(x, csr=csr, aggr=aggr)
        torch.cuda.synchronize()
        ref, _, sabs = oracle.propagate(x_np, ei_np, w_np, aggr=aggr)
        check_sum(out, ref, sabs, False, f"empty runs N={N} E={E} F={F} {aggr}")
    out, arg = pyg.propagate(x, csr=plain, aggr="max")
    torch.cuda.synchronize()
    ref, rarg, _ = oracle.propagate(x_np, ei_np, None, aggr="max")
    check_max(out, arg, ref, rarg, what=f"empty runs N={N} E={E} F={F} max")
    # the blocked form (empty virtual rows as well)
    for B in (2, 8):
        bc = pyg.coo_to_csr_blocked(ei, N, B, with_perm=True)
        outb, argb = pyg.propagate_blocked(x, bc, "max")
        torch.cuda.synchronize()
        check_max(outb, argb, ref, rarg, what=f"empty runs blocked B={B} N={N} E={E} F={F} max")
        outg = pyg.gcn_propagate_blocked(x, None, bc)
        torch.cuda.synchronize()
        w_or = oracle.gcn_norm(ei_np, N).astype(np.float32)
        refg, _, sabsg = oracle.propagate(x_np, ei_np, w_or, aggr="sum")
        check_sum(outg, refg, sabsg, False, f"empty runs blocked gcn B={B} N={N} E={E} F={F}")


@pytest.mark.parametrize("N,E", GRAPHS)
def test_row_walkers_empty_runs(pyg, N, E):
    """gcn_norm in CSR order, the softmax, the weight gradient and the
    attention backward's head dot products on the same graphs."""
    rng = np.random.default_rng(N + 3 * E)
    ei_np = runs_graph(rng, N, E)
    ei = to_dev(ei_np)
    csr = pyg.coo_to_csr(ei, N)
    rp, col, perm = oracle.coo_to_csr(ei_np, N)
    norm = pyg.gcn_norm_csr(csr)
    torch.cuda.synchronize()
    assert np.array_equal(norm.cpu().numpy(), oracle.gcn_norm(ei_np, N).astype(np.float32)[perm])
    H = 4
    s_np = rng.standard_normal((E, H)).astype(np.float32)
    alpha = pyg.segment_softmax(to_dev(s_np), csr, "coo")
    torch.cuda.synchronize()
    check_softmax(alpha, oracle.segment_softmax(s_np, ei_np, N), s_np, ei_np[1], N, f"softmax empty runs E={E}")
    F = 32
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    g_np = rng.standard_normal((N, F)).astype(np.float32)
    w_np = rng.standard_normal(E).astype(np.float32)
    d_w = to_dev(w_np)
    csr_w = pyg.coo_to_csr(ei, N, d_w)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, d_w)
    gx, gw = pyg.propagate_backward(to_dev(g_np), to_dev(x_np), ei, d_w, csr_w, csr_t, "sum", need_grad_w=True)
    torch.cuda.synchronize()
    ref_x, ref_w, sx, sw = oracle.propagate_backward(x_np, ei_np, g_np, w_np, aggr="sum", want_grad_w=True)
    check_sum(gx, ref_x, sx, False, f"backward grad_x empty runs E={E}")
    check_sum(gw, ref_w, sw, False, f"backward grad_w empty runs E={E}")


def test_pool_many_empty_graphs(pyg):
    """A batch in which most graphs have no nodes (long runs of empty rows of
    the pooling's segment walk)."""
    rng = np.random.default_rng(77)
    G, n = 50000, 6000
    batch_np = np.sort(np.concatenate([rng.integers(20000, 21000, n // 2), rng.integers(40000, 40500, n // 2)]))
    x_np = rng.standard_normal((n, 24)).astype(np.float32)
    for aggr in ("sum", "mean", "max"):
        out, arg = pyg.global_pool(to_dev(x_np), to_dev(batch_np), G, aggr)
        torch.cuda.synchronize()
        ref, rarg, sabs = oracle.global_pool(x_np, batch_np, G, aggr)
        if aggr == "max":
            check_max(out, arg, ref, rarg, what="pool max, empty graphs")
        else:
            check_sum(out, ref, sabs, False, f"pool {aggr}, empty graphs")
