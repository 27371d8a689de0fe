"""GPU parity of pyg_gcn_propagate (the GCN normalisation formed per slot
inside the propagate): its norms bit for bit against pyg_gcn_norm_csr and
the oracle's gcn_norm, its output against the oracle's weighted sum."""
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
