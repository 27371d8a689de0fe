"""GPU parity of the attention gradients (attention sum and GAT scores)
against the oracle, per stage on identical inputs, plus a whole GAT layer's
gradient chain."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_sum, to_dev

pytestmark = pytest.mark.gpu

CASES = [(1, 4, 1, 3), (9, 0, 2, 4), (60, 400, 1, 16), (300, 5000, 3, 8), (2000, 30000, 8, 8), (700, 9000, 4, 32),
         (400, 3000, 16, 4), (257, 4000, 2, 130)]


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def graphs(pyg, rng, N, E, chunk=0, hub=False):
    ei = synth.random_coo(rng, N, E)
    if hub and E:
        ei[1, : E // 2] = 0
        ei[0, E // 2:] = 1
    d_ei = to_dev(ei)
    csr = pyg.coo_to_csr(d_ei, N, chunk=chunk)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N, chunk=chunk)
    _, _, perm = oracle.coo_to_csr(ei, N)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)
    return ei, csr, csr_t, perm


def transpose_map_ref(ei, N):
    """The slot of the CSR holding the edge of each slot of the reversed CSR,
    from the oracle's two CSR permutations."""
    _, _, perm = oracle.coo_to_csr(ei, N)
    _, _, perm_t = oracle.coo_to_csr(ei[::-1].copy(), N)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(len(perm))
    return inv[perm_t]


def test_csr_transpose_map(pyg):
    # from 2^20 edges on, the inverse permutation is partitioned by edge id
    # and written block by block: one and two radix passes over the id bits
    # above the 2^14-id LDS blocks, ragged last blocks and tiles
    for i, (N, E) in enumerate([(1, 0), (5, 1), (300, 5000), (3000, 90000), (40000, 1 << 20),
                                (70000, 1_500_001), (300000, 2_200_037)]):
        rng = np.random.default_rng(870 + i)
        ei, csr, csr_t, _ = graphs(pyg, rng, N, E, 64 if i == 3 else 0, hub=i in (3, 6))
        got = pyg.csr_transpose_map(csr, csr_t)
        torch.cuda.synchronize()
        assert got.dtype == torch.int32 and np.array_equal(got.cpu().numpy(), transpose_map_ref(ei, N)), (N, E)


def test_csr_transpose_map_malformed_perm_stays_in_bounds(pyg):
    # a permutation with repeated ids (not one built by coo_to_csr): the map
    # is meaningless but every entry lies in [0, E)
    rng = np.random.default_rng(881)
    N, E = 50000, 1_300_000
    ei, csr, csr_t, _ = graphs(pyg, rng, N, E)
    bad = csr.perm.clone()
    bad[: E // 3] = bad[E // 3: 2 * (E // 3)]
    got = pyg.csr_transpose_map(pyg.CSR(csr.rowptr, csr.col, bad, csr.weight, csr.N, csr.E, csr.chunk), csr_t)
    torch.cuda.synchronize()
    g = got.cpu().numpy()
    assert g.min() >= 0 and g.max() < E


def heads_bwd_case(pyg, N, E, H, C, seed, dtype, chunk=0, hub=False, use_map=False):
    rng = np.random.default_rng(seed)
    ei, csr, csr_t, perm = graphs(pyg, rng, N, E, chunk, hub)
    mt = pyg.csr_transpose_map(csr, csr_t) if use_map else None
    x = rng.standard_normal((N, H * C)).astype(np.float32)
    g = rng.standard_normal((N, H * C)).astype(np.float32)
    if dtype == torch.bfloat16:
        x, g = bf16_round(x), bf16_round(g)
    alpha = rng.random((E, H)).astype(np.float32)
    rx, ra, sx, sa = oracle.propagate_heads_backward(x, ei, alpha, g, H)
    gx, ga = pyg.propagate_heads_backward(to_dev(g).to(dtype), to_dev(x).to(dtype), csr, csr_t, to_dev(alpha[perm]), H,
                                          map_t=mt)
    torch.cuda.synchronize()
    tag = f"heads bwd N={N} E={E} H={H} C={C} {dtype} chunk={chunk}"
    check_sum(gx, rx, sx, dtype == torch.bfloat16, tag + " grad_x")
    ga_coo = np.empty_like(ra)
    if E:
        ga_coo[perm] = ga.cpu().numpy()
    check_sum(torch.from_numpy(ga_coo), ra, sa, False, tag + " grad_alpha")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_propagate_heads_backward(pyg, dtype):
    for i, (N, E, H, C) in enumerate(CASES):
        heads_bwd_case(pyg, N, E, H, C, 900 + i, dtype, use_map=i % 2 == 1)


def test_propagate_heads_backward_shapes(pyg):
    """Head widths on both sides of the vector kernel's conditions: C a
    multiple of the lane vector or not, lanes per head not a power of two
    (C = 24 fp32), heads wider than a wavefront (C = 320 fp32) and rows of
    more than 64 lane vectors (F = 512 fp32, two windows)."""
    for i, (H, C, dtype) in enumerate([(4, 24, torch.float32), (2, 320, torch.float32), (8, 64, torch.float32),
                                       (3, 8, torch.bfloat16), (2, 4, torch.bfloat16), (1, 1, torch.float32),
                                       (16, 32, torch.bfloat16)]):
        heads_bwd_case(pyg, 500, 6000, H, C, 880 + i, dtype, use_map=True)


@pytest.mark.parametrize("chunk", [0, 64])
def test_propagate_heads_backward_hubs(pyg, chunk):
    heads_bwd_case(pyg, 3000, 30000, 8, 8, 31, torch.float32, chunk=chunk, hub=True)
    heads_bwd_case(pyg, 3000, 30000, 8, 16, 32, torch.bfloat16, chunk=chunk, hub=True, use_map=True)


def gat_bwd_case(pyg, N, E, H, seed, slope=0.2, chunk=0, hub=False, use_map=False):
    rng = np.random.default_rng(seed)
    ei, csr, csr_t, perm = graphs(pyg, rng, N, E, chunk, hub)
    mt = pyg.csr_transpose_map(csr, csr_t) if use_map else None
    a_src = rng.standard_normal((N, H)).astype(np.float32)
    a_dst = rng.standard_normal((N, H)).astype(np.float32)
    ge = rng.standard_normal((E, H)).astype(np.float32)
    rs, rd, ss, sd = oracle.gat_scores_backward(a_src, a_dst, ei, ge, slope)
    gs, gd = pyg.gat_scores_backward(to_dev(a_src), to_dev(a_dst), csr, csr_t, to_dev(ge[perm]), slope, map_t=mt)
    torch.cuda.synchronize()
    tag = f"gat bwd N={N} E={E} H={H} chunk={chunk}"
    check_sum(gs, rs, ss, False, tag + " a_src")
    check_sum(gd, rd, sd, False, tag + " a_dst")


def test_gat_scores_backward(pyg):
    for i, (N, E, H, _) in enumerate(CASES):
        gat_bwd_case(pyg, N, E, H, 950 + i, use_map=i % 2 == 0)
    for chunk in (0, 64):
        gat_bwd_case(pyg, 3000, 30000, 8, 32, slope=0.01, chunk=chunk, hub=True, use_map=chunk == 64)


def test_gat_layer_gradients(pyg):
    """Forward (coefficients, attention sum) and backward (attention sum,
    softmax, scores) of one GAT layer on the PubMed-shaped graph, all on the
    GPU, against the oracle chain. The GPU's fp32 coefficients and
    intermediate gradients differ from the oracle's within their own stage
    tolerances; the chain is checked normwise: max |gpu - ref| <= 1e-4 max |ref|."""
    c = synth.make_config(2, F=64)
    N, ei = c["N"], c["edge_index_gcn"]
    H, C = 8, 8
    rng = np.random.default_rng(33)
    x = c["x"]
    a_src = rng.standard_normal((N, H)).astype(np.float32)
    a_dst = rng.standard_normal((N, H)).astype(np.float32)
    g = rng.standard_normal((N, H * C)).astype(np.float32)
    d_ei = to_dev(ei)
    csr = pyg.coo_to_csr(d_ei, N)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(d_ei), N)
    d_src, d_dst, d_x, d_g = to_dev(a_src), to_dev(a_dst), to_dev(x), to_dev(g)
    mt = pyg.csr_transpose_map(csr, csr_t)
    alpha = pyg.gat_softmax(d_src, d_dst, csr, 0.2, "csr")
    gx, galpha = pyg.propagate_heads_backward(d_g, d_x, csr, csr_t, alpha, H, map_t=mt)
    gscore = pyg.segment_softmax_backward(alpha, galpha, csr, "csr")
    gs, gd = pyg.gat_scores_backward(d_src, d_dst, csr, csr_t, gscore, 0.2, map_t=mt)
    torch.cuda.synchronize()
    e = oracle.gat_scores(a_src, a_dst, ei, 0.2)
    al = oracle.segment_softmax(e, ei, N).astype(np.float32)
    rx, ra, _, _ = oracle.propagate_heads_backward(x, ei, al, g, H)
    rsc, _ = oracle.segment_softmax_backward(al, ra.astype(np.float32), ei, N)
    rs, rd, _, _ = oracle.gat_scores_backward(a_src, a_dst, ei, rsc.astype(np.float32), 0.2)
    for got, ref, name in ((gx, rx, "grad_x"), (gs, rs, "grad_a_src"), (gd, rd, "grad_a_dst")):
        err = np.abs(got.cpu().numpy().astype(np.float64) - ref).max()
        assert err <= 1e-4 * np.abs(ref).max() + 1e-6, f"{name}: {err} vs {np.abs(ref).max()}"


def test_attention_backward_is_deterministic(pyg):
    rng = np.random.default_rng(34)
    N, E, H, C = 4000, 90000, 8, 16
    ei, csr, csr_t, _ = graphs(pyg, rng, N, E, 64, hub=True)
    g = torch.randn(N, H * C, device="cuda")
    x = torch.randn(N, H * C, device="cuda")
    alpha = torch.rand(E, H, device="cuda")
    a_s, a_d = torch.randn(N, H, device="cuda"), torch.randn(N, H, device="cuda")
    ge = torch.randn(E, H, device="cuda")
    mt = pyg.csr_transpose_map(csr, csr_t)
    first = pyg.propagate_heads_backward(g, x, csr, csr_t, alpha, H)
    f2 = pyg.gat_scores_backward(a_s, a_d, csr, csr_t, ge)
    for i in range(2):  # with and without the precomputed map: the same bits
        m = mt if i else None
        again = pyg.propagate_heads_backward(g, x, csr, csr_t, alpha, H, map_t=m)
        assert torch.equal(again[0], first[0]) and torch.equal(again[1], first[1])
        a2 = pyg.gat_scores_backward(a_s, a_d, csr, csr_t, ge, map_t=m)
        assert torch.equal(a2[0], f2[0]) and torch.equal(a2[1], f2[1])
