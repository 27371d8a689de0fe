"""GPU parity of propagate with F-dimensional edge features (x_j + e,
max(x_j + e, 0), x_j * e) against the oracle on identical seeded inputs:
both kernels, edge features in COO or CSR slot order, fp32 and bf16."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_max, check_sum, to_dev

pytestmark = pytest.mark.gpu

CASES = [(1, 4, 3), (9, 0, 8), (60, 400, 1), (300, 5000, 16), (2000, 30000, 64), (700, 9000, 128), (400, 3000, 500),
         (257, 4000, 260)]
MSGS = ["edge_add", "edge_relu", "edge_mul"]


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def run_case(pyg, N, E, F, seed, msg, aggr, dtype, kernel, order, chunk=0, hub=False):
    rng = np.random.default_rng(seed)
    ei = synth.random_coo(rng, N, E)
    if hub and E:
        ei[1, : E // 2] = 0
    x = rng.standard_normal((N, F)).astype(np.float32)
    ea = rng.standard_normal((E, F)).astype(np.float32)
    if dtype == torch.bfloat16:
        x, ea = bf16_round(x), bf16_round(ea)
    d_ei = to_dev(ei)
    csr = None
    ea_in = ea
    if kernel == "csr":
        csr = pyg.coo_to_csr(d_ei, N, chunk=chunk)
        if order == "csr":
            _, _, perm = oracle.coo_to_csr(ei, N)
            assert np.array_equal(csr.perm.cpu().numpy(), perm)
            ea_in = ea[perm]
    out, arg = pyg.propagate_edge(to_dev(x).to(dtype), to_dev(ea_in).to(dtype), d_ei, csr, msg, aggr, kernel, order)
    torch.cuda.synchronize()
    ref, rarg, sabs = oracle.propagate(x, ei, msg=msg, aggr=aggr, edge_attr=ea)
    tag = f"edge N={N} E={E} F={F} {msg} {aggr} {dtype} {kernel}/{order} chunk={chunk}"
    if aggr == "max":
        check_max(out, arg, ref, rarg, dtype == torch.bfloat16, tag)
    else:
        check_sum(out, ref, sabs, dtype == torch.bfloat16, tag)


COMBOS = [(m, a, d, k) for m in MSGS for a in ("sum", "mean", "max") for d in (torch.float32, torch.bfloat16)
          for k in (("coo", "coo"), ("csr", "coo"), ("csr", "csr"))]


@pytest.mark.parametrize("msg,aggr,dtype,ko", COMBOS,
                         ids=[f"{m}-{a}-{str(d)[6:]}-{k[0]}{k[1]}" for m, a, d, k in COMBOS])
def test_propagate_edge(pyg, msg, aggr, dtype, ko):
    for i, (N, E, F) in enumerate(CASES):
        run_case(pyg, N, E, F, 700 + i, msg, aggr, dtype, ko[0], ko[1])


@pytest.mark.parametrize("chunk", [0, 64])
@pytest.mark.parametrize("aggr", ["sum", "max"])
def test_propagate_edge_long_rows(pyg, chunk, aggr):
    for msg in MSGS:
        run_case(pyg, 3000, 30000, 32, 21, msg, aggr, torch.float32, "csr", "csr", chunk=chunk, hub=True)
        run_case(pyg, 3000, 30000, 32, 22, msg, aggr, torch.float32, "csr", "coo", chunk=chunk, hub=True)


def test_propagate_edge_light_rows(pyg):
    for msg in MSGS:
        for aggr in ("sum", "max"):
            run_case(pyg, 20000, 60000, 16, 23, msg, aggr, torch.float32, "csr", "csr")


def test_edge_add_zero_is_plain_propagate(pyg):
    """e = 0 must give exactly the plain CSR propagate (values and argmax)."""
    c = synth.make_config(4)
    N, ei, x = c["N"], c["edge_index"], c["x"]
    d_ei, d_x = to_dev(ei), to_dev(x)
    csr = pyg.coo_to_csr(d_ei, N)
    zero = torch.zeros(ei.shape[1], x.shape[1], device="cuda")
    for aggr in ("sum", "max"):
        a, aa = pyg.propagate_edge(d_x, zero, d_ei, csr, "edge_add", aggr, "csr", "csr")
        b, ba = pyg.propagate(d_x, d_ei, csr=csr, aggr=aggr)
        assert torch.equal(a, b)
        if aggr == "max":
            assert torch.equal(aa, ba)
