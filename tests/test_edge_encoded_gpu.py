"""GPU parity of pyg_propagate_edge_encoded (edge features of width D
projected to F by the dense transform, then the edge-feature message)
against the oracle's two steps: oracle.dense_transform, then
oracle.propagate with the projected features. Edge features are small
integers and Theta_e multiples of 1/8, so every projected feature is exact
in fp32 and in bf16 on both sides: the messages are then identical and max /
argmax can be compared bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_max, check_sum, to_dev

pytestmark = pytest.mark.gpu

MSGS = ["edge_add", "edge_relu", "edge_mul"]


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


def inputs(rng, N, E, F, D):
    x = rng.standard_normal((N, F)).astype(np.float32)
    ea = rng.integers(-2, 3, (E, D)).astype(np.float32)
    th = (rng.integers(-4, 5, (D, F)) / 8.0).astype(np.float32)
    return x, ea, th


# (N, E, F, D): D below, equal to and above F, odd widths, no features (D = 0), no edges
CASES = [(300, 5000, 16, 7), (700, 9000, 128, 16), (50, 400, 64, 1), (257, 4000, 32, 0), (400, 3000, 24, 40),
         (9, 0, 8, 4), (2000, 30000, 64, 16)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
def test_edge_encoded(pyg, aggr, dtype):
    bf16 = dtype == torch.bfloat16
    for i, (N, E, F, D) in enumerate(CASES):
        rng = np.random.default_rng(800 + i)
        ei = synth.random_coo(rng, N, E)
        x, ea, th = inputs(rng, N, E, F, D)
        if bf16:
            x = bf16_round(x)
        e, _ = oracle.dense_transform(ea, th) if D else (np.zeros((E, F)), None)
        e32 = e.astype(np.float32)
        assert np.array_equal(e32.astype(np.float64), e)  # exact by construction
        d_ei = to_dev(ei)
        csr = pyg.coo_to_csr(d_ei, N)
        _, _, perm = oracle.coo_to_csr(ei, N)
        for j, msg in enumerate(MSGS):
            ref, rarg, sabs = oracle.propagate(x, ei, msg=msg, aggr=aggr, edge_attr=e32)
            runs = [("csr", "coo", ea), ("csr", "csr", ea[perm] if E else ea)]
            if aggr == "sum" and not bf16:
                runs.append(("coo", "coo", ea))
            for kernel, order, ea_in in runs:
                out, arg = pyg.propagate_edge_encoded(to_dev(x).to(dtype), to_dev(ea_in).to(dtype),
                                                      to_dev(th).to(dtype), d_ei, csr if kernel == "csr" else None,
                                                      msg, aggr, kernel, order)
                torch.cuda.synchronize()
                tag = f"encoded N={N} E={E} F={F} D={D} {msg} {aggr} {kernel} {order} {dtype}"
                if aggr == "max":
                    check_max(out, arg, ref, rarg, bf16, tag)
                else:
                    check_sum(out, ref, sabs, bf16, tag)


def test_edge_encoded_random_theta_sum(pyg):
    """Real-valued features and Theta_e: the projection rounds in fp32, so the
    sum is checked with the sum rule over the messages plus the rounding of
    each projected feature carried through (|x_j| + 1 times D ulps of
    sum_d |e_d theta_d|)."""
    rng = np.random.default_rng(890)
    N, E, F, D = 1500, 20000, 64, 24
    ei = synth.random_coo(rng, N, E)
    x = rng.standard_normal((N, F)).astype(np.float32)
    ea = rng.standard_normal((E, D)).astype(np.float32)
    th = (rng.standard_normal((D, F)) / np.sqrt(D)).astype(np.float32)
    e, es = oracle.dense_transform(ea, th)
    csr = pyg.coo_to_csr(to_dev(ei), N)
    for msg in MSGS:
        ref, _, sabs = oracle.propagate(x, ei, msg=msg, aggr="sum", edge_attr=e.astype(np.float32))
        # per edge the projected feature may differ by up to D + 1 fp32 roundings of es
        slack = np.zeros((N, F))
        np.add.at(slack, ei[1], (np.abs(x[ei[0]]) + 1.0) * es * (D + 1) * 2.0 ** -24)
        out, _ = pyg.propagate_edge_encoded(to_dev(x), to_dev(ea), to_dev(th), to_dev(ei), csr, msg, "sum")
        torch.cuda.synchronize()
        g = out.cpu().numpy().astype(np.float64)
        bound = 1e-5 * sabs + 1e-6 + slack
        assert np.all(np.abs(g - ref) <= bound), f"encoded random {msg}: {np.max(np.abs(g - ref) - bound)}"
