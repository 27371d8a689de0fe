"""GPU parity of the source-blocked propagate path: pyg_csr_blocks_build and
pyg_coo_to_csr_blocked (bit-exact against a stable sort of the oracle's CSR
by source block), pyg_degree_csr_blocks (bit-exact against the oracle's
degree) and pyg_propagate_blocked against the oracle (sum / mean within the
parity rule, max / argmax bit for bit, ties across blocks to the lowest edge
id)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_max, check_sum, to_dev

pytestmark = pytest.mark.gpu

F32, BF16 = torch.float32, torch.bfloat16


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    m.library()
    return m


def expected_blocks(ei_np, N, B, w_np=None):
    """The blocked CSR from the oracle's CSR: slots stably ordered by
    (source block, target), i.e. virtual row b * N + i."""
    rp, col, perm = oracle.coo_to_csr(ei_np, N)
    E = col.shape[0]
    row = np.repeat(np.arange(N), np.diff(rp))
    bsize = -(-N // B) if N else 1
    key = (col // bsize) * N + row
    order = np.argsort(key, kind="stable")
    brp = np.concatenate([[0], np.cumsum(np.bincount(key, minlength=B * N))]).astype(np.int64)
    w = None if w_np is None else w_np[perm][order]
    return brp, col[order], perm[order], w, E


def make(pyg, ei_np, N, B, w_np=None, chunk=0, with_perm=True):
    ei = to_dev(ei_np)
    w = to_dev(w_np) if w_np is not None else None
    csr = pyg.coo_to_csr(ei, N, w, chunk=chunk)
    return pyg.csr_blocks(csr, B, with_perm=with_perm), csr


GRAPHS = [(1, 0), (5, 40), (300, 5000), (2000, 40000), (7001, 90000)]


@pytest.mark.parametrize("N,E", GRAPHS)
@pytest.mark.parametrize("B", [2, 3, 4, 8, 16, 32])
def test_csr_blocks_bit_exact(pyg, N, E, B):
    rng = np.random.default_rng(N + E + B)
    ei_np = synth.random_coo(rng, N, E)
    w_np = rng.standard_normal(E).astype(np.float32)
    bc, _ = make(pyg, ei_np, N, B, w_np)
    torch.cuda.synchronize()
    brp, col, perm, w, _ = expected_blocks(ei_np, N, B, w_np)
    assert np.array_equal(bc.rowptr.cpu().numpy(), brp)
    assert np.array_equal(bc.col.cpu().numpy().astype(np.int64), col)
    assert np.array_equal(bc.perm.cpu().numpy(), perm)
    assert np.array_equal(bc.weight.cpu().numpy(), w)


# the packed sort (key, source and edge id in one 64-bit word) and, for the
# last graph (2 * 21 + 22 + 1 bits), the sort with separate fields
DIRECT = [(1, 0), (5, 40), (300, 5000), (7001, 90000), (2_100_000, 4_200_000)]


@pytest.mark.parametrize("N,E,B", [(3_000_000, 400_000, 2), (1_500_000, 300_000, 4)])
def test_coo_to_csr_blocked_wide_keys(pyg, N, E, B):
    # 23-bit blocked keys, two blocks over 22-bit targets and four over
    # 21-bit ones (packed passes of 5, 6, 6, 6 bits: the 17 bits below the
    # last digit do not fit 2 bytes, so the keys are kept whole as rows)
    rng = np.random.default_rng(N + 3 * E + B)
    ei_np = synth.random_coo(rng, N, E)
    brp, col, perm, _, _ = expected_blocks(ei_np, N, B, None)
    bc = pyg.coo_to_csr_blocked(to_dev(ei_np), N, B, with_perm=True)
    torch.cuda.synchronize()
    assert np.array_equal(bc.rowptr.cpu().numpy(), brp)
    assert np.array_equal(bc.col.cpu().numpy().astype(np.int64), col)
    assert np.array_equal(bc.perm.cpu().numpy(), perm)


@pytest.mark.parametrize("N,E", DIRECT)
@pytest.mark.parametrize("B", [2, 3, 8, 32])
def test_coo_to_csr_blocked_bit_exact(pyg, N, E, B):
    if N > 100_000 and B not in (2, 32):
        pytest.skip("one small and one large block count on the large graph")
    rng = np.random.default_rng(N + E + 7 * B)
    ei_np = synth.random_coo(rng, N, E)
    w_np = rng.standard_normal(E).astype(np.float32)
    ei = to_dev(ei_np)
    brp, col, perm, w, _ = expected_blocks(ei_np, N, B, w_np)
    bc = pyg.coo_to_csr_blocked(ei, N, B, to_dev(w_np), with_perm=True)
    deg = pyg.degree_csr_blocks(bc)
    torch.cuda.synchronize()
    assert np.array_equal(bc.rowptr.cpu().numpy(), brp)
    assert np.array_equal(bc.col.cpu().numpy().astype(np.int64), col)
    assert np.array_equal(bc.perm.cpu().numpy(), perm)
    assert np.array_equal(bc.weight.cpu().numpy(), w)
    assert np.array_equal(deg.cpu().numpy(), oracle.degree(ei_np, N))
    # without weights and edge ids: the same rowptr and columns
    bp = pyg.coo_to_csr_blocked(ei, N, B)
    torch.cuda.synchronize()
    assert bp.perm is None and bp.weight is None
    assert torch.equal(bp.rowptr, bc.rowptr) and torch.equal(bp.col, bc.col)
    # equal to the blocks regrouped from the plain CSR
    if E:
        rg = pyg.csr_blocks(pyg.coo_to_csr(ei, N, to_dev(w_np)), B, with_perm=True)
        torch.cuda.synchronize()
        assert torch.equal(rg.rowptr, bc.rowptr) and torch.equal(rg.col, bc.col) and torch.equal(rg.perm, bc.perm)


def run_case(pyg, ei_np, x_np, B, w_np=None, msg="src", aggr="sum", dtype=F32, chunk=0, what=""):
    N = x_np.shape[0]
    x_in = x_np if dtype == F32 else bf16_round(x_np)
    x = to_dev(x_np).to(dtype)
    bc, _ = make(pyg, ei_np, N, B, w_np, chunk=chunk)
    out, arg = pyg.propagate_blocked(x, bc, aggr=aggr, msg=msg)
    torch.cuda.synchronize()
    ref, rarg, sabs = oracle.propagate(x_in, ei_np, w_np, msg=msg, aggr=aggr)
    tag = f"{what} B={B} {msg} {aggr} {dtype} w={w_np is not None} chunk={chunk}"
    if aggr == "max":
        check_max(out, arg, ref, rarg, dtype == BF16, tag)
    else:
        check_sum(out, ref, sabs, dtype == BF16, tag)
    return out, arg


# (N, E, F): ragged windows (F = 20: one 8-lane window of which 5 lanes work;
# F = 500: 15 full windows and a 5-lane one), a single-vector row (F = 4),
# the large graph's width (F = 128)
SHAPES = [(300, 5000, 4), (700, 9000, 20), (2000, 40000, 128), (400, 6000, 500), (6, 50, 32)]


@pytest.mark.parametrize("N,E,F", SHAPES)
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_propagate_blocked_weighted(pyg, N, E, F, aggr, dtype):
    if dtype == BF16 and (F * 2) % 16 != 0:
        pytest.skip("bf16 rows of F = %d are not 16-byte vectors" % F)
    rng = np.random.default_rng(N * 7 + F)
    ei_np = synth.random_coo(rng, N, E)
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    w_np = rng.standard_normal(E).astype(np.float32)
    run_case(pyg, ei_np, x_np, 8, w_np, aggr=aggr, dtype=dtype, what=f"N={N} E={E} F={F}")


@pytest.mark.parametrize("B", [2, 3, 4, 5, 8, 16, 24, 32])
@pytest.mark.parametrize("msg,aggr", [("src", "sum"), ("src", "max"), ("diff", "mean"), ("diff", "max")])
def test_propagate_blocked_messages_and_blocks(pyg, B, msg, aggr):
    rng = np.random.default_rng(B)
    N, E, F = 3000, 60000, 64
    ei_np = synth.random_coo(rng, N, E)
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    run_case(pyg, ei_np, x_np, B, None, msg=msg, aggr=aggr, what="plain")


@pytest.mark.parametrize("chunk", [16, 64])
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
def test_propagate_blocked_long_rows(pyg, chunk, aggr):
    # hub targets whose virtual rows span many chunks (pieces folded by the
    # fix-up) beside light rows and empty virtual rows
    rng = np.random.default_rng(chunk)
    N, F = 900, 96
    hubs = rng.integers(0, N, 6)
    dst = np.concatenate([np.repeat(hubs, 1500), rng.integers(0, N, 4000)])
    src = rng.integers(0, N, dst.shape[0])
    perm = rng.permutation(dst.shape[0])
    ei_np = np.stack([src[perm], dst[perm]]).astype(np.int64)
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    w_np = rng.standard_normal(ei_np.shape[1]).astype(np.float32)
    for dtype in (F32, BF16):
        for B in (2, 16):
            run_case(pyg, ei_np, x_np, B, w_np, aggr=aggr, dtype=dtype, chunk=chunk, what="hubs")


def test_propagate_blocked_ties_across_blocks(pyg):
    # integer features: equal maxima in several source blocks of one row must
    # resolve to the lowest edge id (and -0.0 ties with +0.0)
    rng = np.random.default_rng(5)
    N, E, F = 1024, 30000, 32
    ei_np = synth.random_coo(rng, N, E)
    x_np = rng.integers(-2, 3, (N, F)).astype(np.float32)
    x_np[rng.random((N, F)) < 0.1] = -0.0
    for B in (2, 8, 32):
        run_case(pyg, ei_np, x_np, B, None, aggr="max", what="ties")
        w_np = rng.integers(-1, 2, E).astype(np.float32)
        run_case(pyg, ei_np, x_np, B, w_np, aggr="max", what="ties weighted")


def test_propagate_blocked_small_and_empty(pyg):
    # fewer nodes than blocks (empty source blocks), no edges at all, isolated targets
    rng = np.random.default_rng(9)
    for N, E in ((3, 7), (5, 0), (40, 3)):
        ei_np = synth.random_coo(rng, N, E) if E else np.zeros((2, 0), np.int64)
        x_np = rng.standard_normal((N, 16)).astype(np.float32)
        for aggr in ("sum", "mean", "max"):
            for B in (2, 8):
                run_case(pyg, ei_np, x_np, B, None, aggr=aggr, what=f"N={N} E={E}")


def test_propagate_blocked_deterministic_and_matches_csr_max(pyg):
    c = synth.make_config(2, seed=0, F=64)
    ei_np, x_np, N = c["edge_index_gcn"], c["x"], c["N"]
    w_np = oracle.gcn_norm(ei_np, N).astype(np.float32)
    ei, x, w = to_dev(ei_np), to_dev(x_np), to_dev(w_np)
    csr = pyg.coo_to_csr(ei, N, w)
    bc = pyg.csr_blocks(csr, 8, with_perm=True)
    a, _ = pyg.propagate_blocked(x, bc, "sum")
    b, _ = pyg.propagate_blocked(x, bc, "sum")
    mb, ab = pyg.propagate_blocked(x, bc, "max")
    mc, ac = pyg.propagate(x, csr=csr, aggr="max")
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32)), "blocked sum is not bit-reproducible"
    assert torch.equal(mb.view(torch.int32), mc.view(torch.int32)) and torch.equal(ab, ac)
    ref, _, sabs = oracle.propagate(x_np, ei_np, w_np, aggr="sum")
    check_sum(a, ref, sabs, False, "PubMed-shaped gcn-weighted sum, blocked")
