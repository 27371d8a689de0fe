"""GPU parity of the attention calls (segment softmax, GAT softmax, their
backward and the multi-head attention sum) against the oracle on identical
seeded inputs."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_softmax, check_sum, to_dev

pytestmark = pytest.mark.gpu

# (N, E, H): chunk-spanning sizes, ragged tails, heads that are not powers of
# two, more heads than lanes (H = 70), an empty edge set
CASES = [(1, 3, 1), (9, 0, 2), (60, 400, 1), (300, 5000, 3), (2000, 30000, 8), (700, 9000, 5),
         (400, 3000, 16), (257, 4000, 70), (5000, 12000, 4)]


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def graph(pyg, rng, N, E, chunk=0, hub=False):
    ei = synth.random_coo(rng, N, E)
    if hub and E:  # one mega-hub target: a row over many chunks
        ei[1, : E // 2] = 0
    d_ei = to_dev(ei)
    csr = pyg.coo_to_csr(d_ei, N, chunk=chunk)
    _, _, perm = oracle.coo_to_csr(ei, N)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)  # slot order is the oracle's (checked, then used)
    return ei, csr, perm


def softmax_case(pyg, N, E, H, seed, order, chunk=0, hub=False, scale=3.0):
    rng = np.random.default_rng(seed)
    ei, csr, perm = graph(pyg, rng, N, E, chunk, hub)
    s = (rng.standard_normal((E, H)) * scale).astype(np.float32)
    ref = oracle.segment_softmax(s, ei, N)
    s_in = s if order == "coo" else s[perm]
    alpha = pyg.segment_softmax(to_dev(s_in), csr, order)
    torch.cuda.synchronize()
    got = alpha.cpu().numpy()
    if order == "csr":
        got = got[np.argsort(perm)] if E else got
    check_softmax(torch.from_numpy(np.ascontiguousarray(got)), ref, s, ei[1], N,
                  f"softmax N={N} E={E} H={H} {order} chunk={chunk} hub={hub}")


@pytest.mark.parametrize("order", ["csr", "coo"])
def test_segment_softmax(pyg, order):
    for i, (N, E, H) in enumerate(CASES):
        softmax_case(pyg, N, E, H, 200 + i, order)


@pytest.mark.parametrize("chunk", [0, 64, 100])
@pytest.mark.parametrize("H", [1, 3, 8])
def test_segment_softmax_long_rows(pyg, chunk, H):
    softmax_case(pyg, 3000, 40000, H, 9, "csr", chunk=chunk, hub=True)
    softmax_case(pyg, 3000, 40000, H, 10, "coo", chunk=chunk, hub=True)


def test_segment_softmax_large_scores(pyg):
    """Scores near 1e3 overflow exp without the segment maximum."""
    for order in ("csr", "coo"):
        softmax_case(pyg, 500, 6000, 4, 11, order, scale=300.0)


def gat_case(pyg, N, E, H, seed, order, slope=0.2, chunk=0, hub=False):
    rng = np.random.default_rng(seed)
    ei, csr, perm = graph(pyg, rng, N, E, chunk, hub)
    a_src = (rng.standard_normal((N, H)) * 2).astype(np.float32)
    a_dst = (rng.standard_normal((N, H)) * 2).astype(np.float32)
    e = oracle.gat_scores(a_src, a_dst, ei, slope)
    ref = oracle.segment_softmax(e, ei, N)
    alpha = pyg.gat_softmax(to_dev(a_src), to_dev(a_dst), csr, slope, order)
    torch.cuda.synchronize()
    got = alpha.cpu().numpy()
    if order == "csr" and E:
        got = got[np.argsort(perm)]
    check_softmax(torch.from_numpy(np.ascontiguousarray(got)), ref, e, ei[1], N,
                  f"gat N={N} E={E} H={H} {order} chunk={chunk}")


@pytest.mark.parametrize("order", ["csr", "coo"])
def test_gat_softmax(pyg, order):
    for i, (N, E, H) in enumerate(CASES):
        gat_case(pyg, N, E, H, 300 + i, order)
    gat_case(pyg, 3000, 40000, 8, 12, order, slope=0.01, chunk=64, hub=True)


def softmax_bwd_case(pyg, N, E, H, seed, order, chunk=0, hub=False):
    rng = np.random.default_rng(seed)
    ei, csr, perm = graph(pyg, rng, N, E, chunk, hub)
    s = (rng.standard_normal((E, H)) * 2).astype(np.float32)
    alpha = oracle.segment_softmax(s, ei, N).astype(np.float32)
    g = rng.standard_normal((E, H)).astype(np.float32)
    ref, sabs = oracle.segment_softmax_backward(alpha, g, ei, N)
    if order == "csr":
        a_in, g_in = alpha[perm], g[perm]
    else:
        a_in, g_in = alpha, g
    gs = pyg.segment_softmax_backward(to_dev(a_in), to_dev(g_in), csr, order)
    torch.cuda.synchronize()
    got = gs.cpu().numpy()
    if order == "csr" and E:
        got = got[np.argsort(perm)]
    err = np.abs(got.astype(np.float64) - ref)
    bound = 1e-5 * sabs + 1e-12
    assert np.all(err <= bound), f"softmax bwd N={N} E={E} H={H} {order}: max err/bound {np.max(err / bound)}"


@pytest.mark.parametrize("order", ["csr", "coo"])
def test_segment_softmax_backward(pyg, order):
    for i, (N, E, H) in enumerate(CASES):
        softmax_bwd_case(pyg, N, E, H, 400 + i, order)
    softmax_bwd_case(pyg, 3000, 40000, 3, 13, order, chunk=64, hub=True)


def heads_case(pyg, N, E, H, C, seed, dtype, chunk=0, hub=False):
    rng = np.random.default_rng(seed)
    ei, csr, perm = graph(pyg, rng, N, E, chunk, hub)
    x = rng.standard_normal((N, H * C)).astype(np.float32)
    if dtype == torch.bfloat16:
        x = bf16_round(x)
    alpha = rng.random((E, H)).astype(np.float32)
    ref, sabs = oracle.propagate_heads(x, ei, alpha, H)
    out = pyg.propagate_heads(to_dev(x).to(dtype), csr, to_dev(alpha[perm]), H)
    torch.cuda.synchronize()
    check_sum(out, ref, sabs, dtype == torch.bfloat16, f"heads N={N} E={E} H={H} C={C} {dtype} chunk={chunk}")


HEAD_SHAPES = [(1, 16), (2, 4), (3, 8), (4, 2), (8, 8), (8, 16), (5, 1), (16, 64)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_propagate_heads(pyg, dtype):
    for i, (N, E, _) in enumerate(CASES[:7]):
        for j, (H, C) in enumerate(HEAD_SHAPES):
            heads_case(pyg, N, E, H, C, 500 + 10 * i + j, dtype)


@pytest.mark.parametrize("chunk", [0, 64])
def test_propagate_heads_long_rows(pyg, chunk):
    for H, C in ((8, 8), (3, 4), (2, 64)):
        heads_case(pyg, 3000, 40000, H, C, 14, torch.float32, chunk=chunk, hub=True)


def test_propagate_heads_light_rows(pyg):
    """Mean degree <= 8 takes the one-row-per-sub-group path."""
    for H, C in ((1, 16), (4, 4), (2, 8)):
        heads_case(pyg, 20000, 60000, H, C, 15, torch.float32)


def test_gat_layer_chain(pyg):
    """GAT attention end to end: coefficients from node logits, then the
    attention sum, against the oracle's chain (fp32 alpha from the oracle).
    Tolerance 2e-5 S + 1e-6: the softmax's own 1e-5 relative error carried
    through the sum, plus the sum's rounding."""
    rng = np.random.default_rng(16)
    c = synth.make_config(2, F=64)
    N, ei = c["N"], c["edge_index_gcn"]
    H, C = 8, 8
    x = c["x"]
    a_src = rng.standard_normal((N, H)).astype(np.float32)
    a_dst = rng.standard_normal((N, H)).astype(np.float32)
    csr = pyg.coo_to_csr(to_dev(ei), N)
    alpha = pyg.gat_softmax(to_dev(a_src), to_dev(a_dst), csr, 0.2, "csr")
    out = pyg.propagate_heads(to_dev(x), csr, alpha, H)
    torch.cuda.synchronize()
    e = oracle.gat_scores(a_src, a_dst, ei, 0.2)
    ref_alpha = oracle.segment_softmax(e, ei, N).astype(np.float32)
    ref, sabs = oracle.propagate_heads(x, ei, ref_alpha, H)
    g = out.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(g - ref) <= 2e-5 * sabs + 1e-6)


def graded_graph(pyg, rng, n_targets, dmax, chunk):
    """Row lengths from 1 to dmax slots in geometric steps (rows that fit a
    group's registers, rows just above, and rows up to a chunk that take the
    two-pass path), a CSR built with the given chunk so that rows up to a
    chunk stay whole."""
    deg = np.unique(np.geomspace(1, dmax, n_targets).astype(np.int64))
    N = max(int(deg.size), 64)
    ei = synth.graded_in_degree(rng, N, deg)
    d_ei = to_dev(ei)
    csr = pyg.coo_to_csr(d_ei, N, chunk=chunk)
    _, _, perm = oracle.coo_to_csr(ei, N)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)
    return ei, csr, perm, N


GRADED = [(4, 6000, 8192), (8, 4096, 4096), (16, 2048, 2048), (64, 300, 1024), (256, 80, 512)]


@pytest.mark.parametrize("H,dmax,chunk", GRADED)
def test_softmax_graded_rows(pyg, H, dmax, chunk):
    """Row lengths across the register path and the two-pass path, whole
    rows up to a chunk: forward from scores in both orders, the fused GAT
    form and the backward, against the oracle."""
    rng = np.random.default_rng(1000 + H)
    ei, csr, perm, N = graded_graph(pyg, rng, 120, dmax, chunk)
    E = ei.shape[1]
    inv = np.argsort(perm)
    s = (rng.standard_normal((E, H)) * 3).astype(np.float32)
    ref = oracle.segment_softmax(s, ei, N)
    for order in ("csr", "coo"):
        got = pyg.segment_softmax(to_dev(s[perm] if order == "csr" else s), csr, order).cpu().numpy()
        got = got[inv] if order == "csr" else got
        check_softmax(torch.from_numpy(np.ascontiguousarray(got)), ref, s, ei[1], N, f"graded softmax H={H} {order}")
    a_src = (rng.standard_normal((N, H)) * 2).astype(np.float32)
    a_dst = (rng.standard_normal((N, H)) * 2).astype(np.float32)
    e = oracle.gat_scores(a_src, a_dst, ei, 0.2)
    got = pyg.gat_softmax(to_dev(a_src), to_dev(a_dst), csr, 0.2, "csr").cpu().numpy()[inv]
    check_softmax(torch.from_numpy(np.ascontiguousarray(got)), oracle.segment_softmax(e, ei, N), e, ei[1], N,
                  f"graded gat H={H}")
    alpha = ref.astype(np.float32)
    g = rng.standard_normal((E, H)).astype(np.float32)
    rb, sabs = oracle.segment_softmax_backward(alpha, g, ei, N)
    for order in ("csr", "coo"):
        a_in, g_in = (alpha[perm], g[perm]) if order == "csr" else (alpha, g)
        got = pyg.segment_softmax_backward(to_dev(a_in), to_dev(g_in), csr, order).cpu().numpy()
        got = got[inv] if order == "csr" else got
        err = np.abs(got.astype(np.float64) - rb)
        bound = 1e-5 * sabs + 1e-12
        assert np.all(err <= bound), f"graded softmax bwd H={H} {order}: max err/bound {np.max(err / bound)}"


def test_softmax_graded_rows_deterministic(pyg):
    rng = np.random.default_rng(1099)
    ei, csr, perm, N = graded_graph(pyg, rng, 150, 4096, 4096)
    E, H = ei.shape[1], 8
    a_src, a_dst = torch.randn(N, H, device="cuda"), torch.randn(N, H, device="cuda")
    s, g = torch.randn(E, H, device="cuda"), torch.randn(E, H, device="cuda")
    first = (pyg.gat_softmax(a_src, a_dst, csr), pyg.segment_softmax(s, csr),
             pyg.segment_softmax_backward(s.softmax(1).contiguous(), g, csr))
    for _ in range(2):
        again = (pyg.gat_softmax(a_src, a_dst, csr), pyg.segment_softmax(s, csr),
                 pyg.segment_softmax_backward(s.softmax(1).contiguous(), g, csr))
        for x, y in zip(first, again):
            assert torch.equal(x, y)


def test_attention_is_deterministic(pyg):
    rng = np.random.default_rng(17)
    N, E, H = 4000, 90000, 8
    ei, csr, _ = graph(pyg, rng, N, E, 64, hub=True)
    a_src = torch.randn(N, H, device="cuda")
    a_dst = torch.randn(N, H, device="cuda")
    x = torch.randn(N, H * 16, device="cuda")
    first = pyg.gat_softmax(a_src, a_dst, csr)
    out = pyg.propagate_heads(x, csr, first, H)
    for _ in range(3):
        again = pyg.gat_softmax(a_src, a_dst, csr)
        assert torch.equal(again, first)
        assert torch.equal(pyg.propagate_heads(x, csr, again, H), out)
