"""GPU parity of pyg_gcn_propagate and pyg_gcn_propagate_blocked (the GCN
normalisation formed per slot inside the propagate, over the CSR or its
source-blocked form): the norms bit for bit against pyg_gcn_norm_csr and the
oracle's gcn_norm, the output against the oracle's weighted sum."""
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


# (N, E, F): light rows (mean degree <= 16), long rows, vector and scalar
# rows, rows wider than one launch (F = 1100: several whole-row launches),
# narrow feature windows (F = 128 at 20k nodes: rows total >= 16 MB)
SHAPES = [(50, 300, 16), (300, 5000, 7), (2000, 40000, 16), (700, 9000, 128), (400, 3000, 500),
          (64, 2000, 1100), (33000, 200000, 128), (5000, 1000, 64)]


@pytest.mark.parametrize("N,E,F", SHAPES)
@pytest.mark.parametrize("weighted", [False, True])
def test_gcn_propagate_parity(pyg, N, E, F, weighted):
    rng = np.random.default_rng(N + E + F)
    ei_np = synth.random_coo(rng, N, E)
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    w_np = (np.abs(rng.standard_normal(E)) + 0.1).astype(np.float32) if weighted else None
    ei = to_dev(ei_np)
    csr = pyg.coo_to_csr(ei, N, to_dev(w_np) if weighted else None)
    norm = torch.full((E,), float("nan"), device="cuda")
    out = pyg.gcn_propagate(to_dev(x_np), csr, norm_out=norm)
    ref_norm = pyg.gcn_norm_csr(csr)
    torch.cuda.synchronize()
    assert torch.equal(norm.view(torch.int32), ref_norm.view(torch.int32)), "norms differ from pyg_gcn_norm_csr"
    rp, col, perm = oracle.coo_to_csr(ei_np, N)
    w_or = oracle.gcn_norm(ei_np, N, w_np).astype(np.float32)
    got = norm.cpu().numpy()
    if not weighted:  # every fp64 step is order-independent: equal to the rounded oracle
        assert np.array_equal(got, w_or[perm])
    else:  # the weighted degree sums in another order: at most one fp32 ulp
        assert np.all(np.abs(got.view(np.int32).astype(np.int64) - w_or[perm].view(np.int32).astype(np.int64)) <= 1)
    ref, _, sabs = oracle.propagate(x_np, ei_np, w_or, aggr="sum")
    check_sum(out, ref, sabs, False, f"gcn_propagate N={N} E={E} F={F} weighted={weighted}")
    # bf16 rows: the same norms, one rounding of the fp32 sum
    if (F * 2) % 16 == 0:
        outb = pyg.gcn_propagate(to_dev(x_np).to(torch.bfloat16), csr)
        torch.cuda.synchronize()
        refb, _, sabsb = oracle.propagate(bf16_round(x_np), ei_np, w_or, aggr="sum")
        check_sum(outb, refb, sabsb, True, f"gcn_propagate bf16 N={N} E={E} F={F}")


def test_gcn_propagate_degenerate(pyg):
    rng = np.random.default_rng(3)
    ei_np = synth.random_coo(rng, 40, 200)
    ei = to_dev(ei_np)
    csr = pyg.coo_to_csr(ei, 40)
    # no features: the norms are still written
    norm = torch.zeros(200, device="cuda")
    pyg.gcn_propagate(torch.empty((40, 0), device="cuda"), csr, norm_out=norm)
    torch.cuda.synchronize()
    assert torch.equal(norm, pyg.gcn_norm_csr(csr))
    # no edges: zeros
    csr0 = pyg.coo_to_csr(torch.zeros((2, 0), dtype=torch.int64, device="cuda"), 40)
    out = pyg.gcn_propagate(to_dev(rng.standard_normal((40, 8)).astype(np.float32)), csr0,
                            norm_out=torch.empty(0, device="cuda"))
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0


BLOCKED_SHAPES = [(50, 300, 16), (300, 5000, 8), (2000, 40000, 16), (700, 9000, 128), (400, 3000, 500),
                  (33000, 200000, 128), (5000, 1000, 64)]


@pytest.mark.parametrize("N,E,F", BLOCKED_SHAPES)
@pytest.mark.parametrize("B", [2, 3, 8])
@pytest.mark.parametrize("weighted", [False, True])
def test_gcn_propagate_blocked_parity(pyg, N, E, F, B, weighted):
    rng = np.random.default_rng(N + E + F + B)
    ei_np = synth.random_coo(rng, N, E)
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    w_np = (np.abs(rng.standard_normal(E)) + 0.1).astype(np.float32) if weighted else None
    ei = to_dev(ei_np)
    csr = pyg.coo_to_csr(ei, N, to_dev(w_np) if weighted else None)
    bc = pyg.csr_blocks(csr, B)
    norm = torch.full((E,), float("nan"), device="cuda")
    out = pyg.gcn_propagate_blocked(to_dev(x_np), csr, bc, norm_out=norm)
    # the reference norms (CSR order) carried into the blocked slot order
    ref_csr = pyg.CSR(csr.rowptr, csr.col, csr.perm, pyg.gcn_norm_csr(csr), N, E, csr.chunk)
    ref_blk = pyg.csr_blocks(ref_csr, B).weight
    torch.cuda.synchronize()
    assert torch.equal(norm.view(torch.int32), ref_blk.view(torch.int32)), "blocked norms differ from pyg_gcn_norm_csr"
    w_or = oracle.gcn_norm(ei_np, N, w_np).astype(np.float32)
    ref, _, sabs = oracle.propagate(x_np, ei_np, w_or, aggr="sum")
    check_sum(out, ref, sabs, False, f"gcn_propagate_blocked B={B} N={N} E={E} F={F} weighted={weighted}")
    # no norm_out: fp32 rows take every window pre-scaled (no norm formed)
    out2 = pyg.gcn_propagate_blocked(to_dev(x_np), csr, bc)
    torch.cuda.synchronize()
    check_sum(out2, ref, sabs, False, f"gcn_propagate_blocked no norms B={B} N={N} E={E} F={F} w={weighted}")
    # bf16 rows (when they are 16-byte vectors): window 0 forms the norms into the workspace
    if (F * 2) % 16 != 0:
        return
    outb = pyg.gcn_propagate_blocked(to_dev(x_np).to(torch.bfloat16), csr, bc)
    torch.cuda.synchronize()
    refb, _, sabsb = oracle.propagate(bf16_round(x_np), ei_np, w_or, aggr="sum")
    check_sum(outb, refb, sabsb, True, f"gcn_propagate_blocked bf16 B={B} N={N} E={E} F={F}")


def test_gcn_propagate_blocked_degenerate(pyg):
    rng = np.random.default_rng(4)
    ei_np = synth.random_coo(rng, 40, 200)
    csr = pyg.coo_to_csr(to_dev(ei_np), 40)
    bc = pyg.csr_blocks(csr, 4)
    # no features: the norms alone, in the blocked order
    norm = torch.zeros(200, device="cuda")
    pyg.gcn_propagate_blocked(torch.empty((40, 0), device="cuda"), csr, bc, norm_out=norm)
    ref = pyg.csr_blocks(pyg.CSR(csr.rowptr, csr.col, csr.perm, pyg.gcn_norm_csr(csr), 40, 200, 0), 4).weight
    torch.cuda.synchronize()
    assert torch.equal(norm, ref)
    # no edges: zeros
    csr0 = pyg.coo_to_csr(torch.zeros((2, 0), dtype=torch.int64, device="cuda"), 40)
    out = pyg.gcn_propagate_blocked(to_dev(rng.standard_normal((40, 8)).astype(np.float32)), csr0,
                                    pyg.csr_blocks(csr0, 2), norm_out=torch.empty(0, device="cuda"))
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0
    # fewer nodes than blocks: empty source blocks
    ei3 = synth.random_coo(rng, 3, 9)
    csr3 = pyg.coo_to_csr(to_dev(ei3), 3)
    x3 = rng.standard_normal((3, 4)).astype(np.float32)
    out3 = pyg.gcn_propagate_blocked(to_dev(x3), csr3, pyg.csr_blocks(csr3, 8))
    torch.cuda.synchronize()
    ref3, _, sabs3 = oracle.propagate(x3, ei3, oracle.gcn_norm(ei3, 3).astype(np.float32), aggr="sum")
    check_sum(out3, ref3, sabs3, False, "gcn_propagate_blocked N=3 B=8")


@pytest.mark.parametrize("N,E,F", [(300, 5000, 8), (2000, 40000, 16), (33000, 200000, 128)])
@pytest.mark.parametrize("weighted", [False, True])
def test_gcn_propagate_blocked_degree_from_blocks(pyg, N, E, F, weighted):
    """d taken from the blocked CSR itself (no plain CSR), built straight from
    the COO: unit weights give the same norms bit for bit; weights sum in
    another fp64 order (at most one fp32 ulp from the oracle's)."""
    rng = np.random.default_rng(N + 3 * E + F)
    ei_np = synth.random_coo(rng, N, E)
    x_np = rng.standard_normal((N, F)).astype(np.float32)
    w_np = (np.abs(rng.standard_normal(E)) + 0.1).astype(np.float32) if weighted else None
    bc = pyg.coo_to_csr_blocked(to_dev(ei_np), N, 2, to_dev(w_np) if weighted else None, with_perm=True)
    norm = torch.full((E,), float("nan"), device="cuda")
    out = pyg.gcn_propagate_blocked(to_dev(x_np), None, bc, norm_out=norm)
    torch.cuda.synchronize()
    w_or = oracle.gcn_norm(ei_np, N, w_np).astype(np.float32)
    exp = w_or[bc.perm.cpu().numpy()]
    got = norm.cpu().numpy()
    if not weighted:
        assert np.array_equal(got, exp)
    else:
        assert np.all(np.abs(got.view(np.int32).astype(np.int64) - exp.view(np.int32).astype(np.int64)) <= 1)
    ref, _, sabs = oracle.propagate(x_np, ei_np, w_or, aggr="sum")
    check_sum(out, ref, sabs, False, f"gcn_propagate_blocked (d from blocks) N={N} E={E} F={F} w={weighted}")
    out2 = pyg.gcn_propagate_blocked(to_dev(x_np), None, bc)
    torch.cuda.synchronize()
    check_sum(out2, ref, sabs, False, f"gcn_propagate_blocked (d from blocks, no norms) N={N} E={E} F={F}")
