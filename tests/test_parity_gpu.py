"""GPU parity: every C-ABI entry point against the oracle on identical seeded
inputs (small graphs that span several chunks and ragged tails, the edge
cases of the method, and the full-size workloads)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_max, check_sum, run_propagate_case, to_dev

pytestmark = pytest.mark.gpu

F32, BF16 = torch.float32, torch.bfloat16


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    m.library()  # raises LibraryMissing when the HIP library was not built
    return m


def graph(N, E, seed, F):
    rng = np.random.default_rng(seed)
    ei = synth.random_coo(rng, N, E)
    x = rng.standard_normal((N, F)).astype(np.float32)
    w = rng.standard_normal(E).astype(np.float32)
    return ei, x, w


# (N, E, F): chunk-spanning sizes with ragged tails, odd and wide feature counts
SMALL = [(1, 0, 4), (1, 5, 3), (7, 0, 16), (50, 300, 1), (300, 5000, 7), (2000, 40000, 16),
         (5000, 1000, 64), (700, 9000, 128), (400, 3000, 500), (64, 2000, 1100), (333, 4444, 260)]


def test_stream_round_trip(pyg):
    ei = to_dev(np.array([[0, 1, 2, 2], [1, 1, 0, 2]], np.int64))
    deg = pyg.degree(ei, 3)
    assert deg.cpu().tolist() == [1, 2, 1]


@pytest.mark.parametrize("N,E,F", SMALL)
def test_degree_and_csr_bit_exact(pyg, N, E, F):
    ei_np, _, w_np = graph(N, E, 1, F)
    ei = to_dev(ei_np)
    assert np.array_equal(pyg.degree(ei, N).cpu().numpy(), oracle.degree(ei_np, N))
    csr = pyg.coo_to_csr(ei, N, to_dev(w_np))
    rp, col, perm = oracle.coo_to_csr(ei_np, N)
    assert np.array_equal(csr.rowptr.cpu().numpy(), rp)
    assert np.array_equal(csr.col.cpu().numpy().astype(np.int64), col)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)
    assert np.array_equal(csr.weight.cpu().numpy(), w_np[perm])
    assert np.array_equal(pyg.degree_csr(csr).cpu().numpy(), oracle.degree(ei_np, N))


def test_csr_many_digits(pyg):
    # N > 2^16 forces three radix passes; heavy duplication tests stability
    rng = np.random.default_rng(3)
    N, E = 300_000, 400_000
    ei_np = np.stack([rng.integers(0, N, E), rng.integers(0, 64, E) * 4099 % N]).astype(np.int64)
    csr = pyg.coo_to_csr(to_dev(ei_np), N)
    rp, col, perm = oracle.coo_to_csr(ei_np, N)
    assert np.array_equal(csr.rowptr.cpu().numpy(), rp)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)
    assert np.array_equal(csr.col.cpu().numpy().astype(np.int64), col)


@pytest.mark.parametrize("N,E", [(2_000_000, 300_000), (3_000_000, 300_000), (6_000_000, 200_000)])
def test_csr_wide_keys(pyg, N, E):
    # packed sorts of 21-bit targets (three passes, the sorted keys' low 14
    # bits kept as 2 bytes), 22-bit targets (four passes of 5, 5, 6, 6 bits:
    # low 16 bits, still 2 bytes) and 23-bit targets (5, 6, 6, 6: low 17 bits,
    # the keys kept whole as rows)
    rng = np.random.default_rng(N + E)
    ei_np = np.stack([rng.integers(0, N, E), rng.integers(0, N, E)]).astype(np.int64)
    ei_np[1, : E // 4] = ei_np[1, : E // 4] % 97  # a few hubs among the spread targets
    csr = pyg.coo_to_csr(to_dev(ei_np), N)
    rp, col, perm = oracle.coo_to_csr(ei_np, N)
    assert np.array_equal(csr.rowptr.cpu().numpy(), rp)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)
    assert np.array_equal(csr.col.cpu().numpy().astype(np.int64), col)


@pytest.mark.parametrize("N,E,F", SMALL)
@pytest.mark.parametrize("weighted", [False, True])
def test_gcn_norm(pyg, N, E, F, weighted):
    ei_np, _, w_np = graph(N, E, 2, F)
    ei_np = synth.with_self_loops(ei_np, N)
    w = np.abs(w_np).astype(np.float32) + np.float32(0.5)
    w = np.concatenate([w, np.ones(N, np.float32)]) if weighted else None
    got = pyg.gcn_norm(to_dev(ei_np), N, to_dev(w) if weighted else None).cpu().numpy()
    ref = oracle.gcn_norm(ei_np, N, w)
    ref32 = ref.astype(np.float32)
    if weighted:  # fp64 degree sums in a different order: at most one fp32 ulp
        ulp = np.spacing(np.abs(ref32))
        assert (np.abs(got.astype(np.float64) - ref) <= ulp).all()
    else:         # every fp64 step is exact-order: bit-identical to the rounded oracle
        assert np.array_equal(got, ref32)
        # the same with the in-degree handed over from pyg_degree
        d_ei = to_dev(ei_np)
        got2 = pyg.gcn_norm(d_ei, N, deg=pyg.degree(d_ei, N)).cpu().numpy()
        assert np.array_equal(got2, ref32)


@pytest.mark.parametrize("N,E,F", SMALL)
@pytest.mark.parametrize("weighted", [False, True])
def test_gcn_norm_csr(pyg, N, E, F, weighted):
    ei_np, _, w_np = graph(N, E, 3, F)
    ei_np = synth.with_self_loops(ei_np, N)
    w = np.concatenate([np.abs(w_np) + np.float32(0.5), np.ones(N, np.float32)]) if weighted else None
    csr = pyg.coo_to_csr(to_dev(ei_np), N, to_dev(w) if weighted else None)
    got = pyg.gcn_norm_csr(csr).cpu().numpy()
    _, _, perm = oracle.coo_to_csr(ei_np, N)
    ref = oracle.gcn_norm(ei_np, N, w)[perm]
    if weighted:  # per-row fp64 sums in another order than the oracle's: at most one fp32 ulp
        assert (np.abs(got.astype(np.float64) - ref) <= np.spacing(np.abs(ref.astype(np.float32)))).all()
    else:
        assert np.array_equal(got, ref.astype(np.float32))


@pytest.mark.parametrize("weighted", [False, True])
def test_gcn_norm_csr_light_rows_with_hubs(pyg, weighted):
    """Short rows on average (the lane-per-row path) with two hub targets of
    5,000 and 700 edges spanning many 64-slot chunks, and empty rows."""
    rng = np.random.default_rng(31)
    N, E = 4000, 20000
    ei_np = synth.random_coo(rng, N, E)
    ei_np[1, :5000] = 7
    ei_np[1, 5000:5700] = N - 1
    ei_np[1, ei_np[1] % 97 == 3] = 8  # some targets lose all their edges (no self-loops: empty rows, d = 0)
    E2 = ei_np.shape[1]
    assert E2 <= 16 * N
    w = (rng.random(E2) + 0.5).astype(np.float32) if weighted else None
    csr = pyg.coo_to_csr(to_dev(ei_np), N, to_dev(w) if weighted else None)
    got = pyg.gcn_norm_csr(csr).cpu().numpy()
    _, _, perm = oracle.coo_to_csr(ei_np, N)
    ref = oracle.gcn_norm(ei_np, N, w)[perm]
    if weighted:
        assert (np.abs(got.astype(np.float64) - ref) <= np.spacing(np.abs(ref.astype(np.float32)))).all()
    else:
        assert np.array_equal(got, ref.astype(np.float32))


COMBOS = [(aggr, msg, kernel, dt) for aggr in ("sum", "mean", "max") for msg in ("src", "weighted", "diff")
          for kernel in ("coo", "csr") for dt in (F32, BF16)]


@pytest.mark.parametrize("aggr,msg,kernel,dtype", COMBOS, ids=[f"{a}-{m}-{k}-{str(d)[6:]}" for a, m, k, d in COMBOS])
def test_propagate_small(pyg, aggr, msg, kernel, dtype):
    for i, (N, E, F) in enumerate(SMALL):
        ei, x, w = graph(N, E, 10 + i, F)
        run_propagate_case(pyg, ei, x, w if msg == "weighted" else None, "diff" if msg == "diff" else "src",
                           aggr, kernel, dtype, what=f"N={N} E={E} F={F}")


@pytest.mark.parametrize("chunk", [64, 100, 256])
@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_long_rows_split_across_chunks(pyg, chunk, aggr, dtype):
    rng = np.random.default_rng(chunk)
    # a mega-hub (in-degree 4999), a power-law graph and hubs that end exactly on chunk edges
    star = synth.star_graph(5000, hub=17, rng=rng)
    pl = synth.symmetrize(synth.chung_lu_pairs(3000, 20000, 2.1, rng))
    exact = np.stack([np.arange(4 * chunk) % 50, np.repeat([3, 9, 9, 9], chunk)]).astype(np.int64)
    for ei, N, F in ((star, 5000, 16), (pl, 3000, 64), (exact, 50, 8), (pl, 3000, 3)):
        x = rng.standard_normal((N, F)).astype(np.float32)
        w = rng.standard_normal(ei.shape[1]).astype(np.float32)
        for wt in (None, w):
            for msg in ("src", "diff"):
                if msg == "diff" and wt is not None:
                    continue
                run_propagate_case(pyg, ei, x, wt, msg, aggr, "csr", dtype, chunk=chunk, what=f"split N={N}")


def test_edge_cases(pyg):
    rng = np.random.default_rng(5)
    # no edges at all
    x = rng.standard_normal((9, 8)).astype(np.float32)
    empty = np.zeros((2, 0), np.int64)
    for kernel in ("coo", "csr"):
        for aggr in ("sum", "mean", "max"):
            run_propagate_case(pyg, empty, x, None, "src", aggr, kernel, what="E=0")
    # all nodes isolated except one self-loop, N = 1 graph
    run_propagate_case(pyg, np.array([[0], [0]], np.int64), x[:1], None, "src", "max", "csr", what="N=1")
    # duplicated edges and exact ties in quantised features, signed zeros
    N, E, F = 40, 2000, 12
    ei = synth.random_coo(rng, N, E)
    ei = np.concatenate([ei, ei[:, :300]], axis=1)
    xq = (np.round(rng.standard_normal((N, F)) * 2) / 2).astype(np.float32)
    xq[xq == 0] = -0.0
    xq[::3, ::2] = 0.0
    wq = (np.round(rng.standard_normal(ei.shape[1]) * 2) / 2).astype(np.float32)
    for kernel in ("coo", "csr"):
        for dt in (F32, BF16):
            for wt in (None, wq):
                run_propagate_case(pyg, ei, xq, wt, "src", "max", kernel, dt, what="ties")
            run_propagate_case(pyg, ei, xq, None, "diff", "max", kernel, dt, what="ties-diff")


def test_max_output_has_no_negative_zero(pyg):
    x = np.array([[-0.0], [0.0], [-1.0]], np.float32)
    ei = np.array([[0, 1, 2], [2, 2, 0]], np.int64)
    for kernel in ("coo", "csr"):
        out, arg = pyg.propagate(to_dev(x), to_dev(ei), csr=pyg.coo_to_csr(to_dev(ei), 3) if kernel == "csr" else None,
                                 aggr="max", kernel=kernel)
        o = out.cpu().numpy()
        assert not np.signbit(o[2, 0]) and arg.cpu().numpy()[2, 0] == 0 and arg.cpu().numpy()[1, 0] == 3


def test_csr_and_max_are_deterministic(pyg):
    c = synth.make_config(2, F=64)
    ei = to_dev(c["edge_index_gcn"])
    x = to_dev(c["x64"])
    N = c["N"]
    norm = pyg.gcn_norm(ei, N)
    csr = pyg.coo_to_csr(ei, N, norm, chunk=64)
    first = pyg.propagate(x, ei, norm, csr=csr, aggr="sum")[0].clone()
    firstmax = pyg.propagate(x, ei, kernel="coo", aggr="max")
    for _ in range(4):
        assert torch.equal(pyg.propagate(x, ei, norm, csr=csr, aggr="sum")[0], first)
        m, a = pyg.propagate(x, ei, kernel="coo", aggr="max")
        assert torch.equal(m, firstmax[0]) and torch.equal(a, firstmax[1])


def test_permutation_invariance(pyg):
    # a simple graph (no duplicate edges) with continuous features has no ties,
    # so the winning edge must map through the permutation
    rng = np.random.default_rng(8)
    ei = synth.random_coo(rng, 500, 6000, duplicates=False)
    x = rng.standard_normal((500, 32)).astype(np.float32)
    p = rng.permutation(ei.shape[1])
    for kernel in ("coo", "csr"):
        m1, a1 = pyg.propagate(to_dev(x), to_dev(ei), kernel=kernel, aggr="max",
                               csr=pyg.coo_to_csr(to_dev(ei), 500) if kernel == "csr" else None)
        m2, a2 = pyg.propagate(to_dev(x), to_dev(ei[:, p]), kernel=kernel, aggr="max",
                               csr=pyg.coo_to_csr(to_dev(ei[:, p]), 500) if kernel == "csr" else None)
        assert torch.equal(m1, m2)
        a1, a2 = a1.cpu().numpy(), a2.cpu().numpy()
        has = a2 < ei.shape[1]
        assert np.array_equal(p[a2[has]], a1[has])


# ------------------------------------------------------------- pooling

@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_global_pool(pyg, aggr, dtype):
    rng = np.random.default_rng(21)
    cases = [((3, 0, 4, 1, 0), 5), ((1,), 64), ((0, 0, 7), 16), (tuple(rng.integers(0, 60, 300)), 128),
             ((5000,), 260)]
    for sizes, F in cases:
        B = len(sizes)
        batch = np.repeat(np.arange(B), sizes).astype(np.int64)
        N = batch.size
        x = rng.standard_normal((N, F)).astype(np.float32)
        xin = x if dtype == F32 else bf16_round(x)
        out, arg = pyg.global_pool(to_dev(x).to(dtype), to_dev(batch), B, aggr)
        ref, rarg, sabs = oracle.global_pool(xin, batch, B, aggr)
        if aggr == "max":
            check_max(out, arg, ref, rarg, dtype == BF16, f"pool {sizes[:5]}")
        else:
            check_sum(out, ref, sabs, dtype == BF16, f"pool {sizes[:5]}")


@pytest.mark.parametrize("aggr", ["sum", "mean", "max"])
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_global_pool_long_graphs_grouped_fold(pyg, aggr, dtype):
    # graphs of many chunks: their pieces are folded in groups first, then
    # the groups' partials in order; small integer features make the maxima
    # tie across many nodes and groups (argmax: the lowest node id)
    rng = np.random.default_rng(23)
    for sizes, F in (((20000,), 8), ((9000, 3, 30000), 5), ((4100,), 130)):
        B = len(sizes)
        batch = np.repeat(np.arange(B), sizes).astype(np.int64)
        N = batch.size
        x = rng.integers(-3, 4, (N, F)).astype(np.float32)
        out, arg = pyg.global_pool(to_dev(x).to(dtype), to_dev(batch), B, aggr)
        ref, rarg, sabs = oracle.global_pool(x, batch, B, aggr)
        if aggr == "max":
            check_max(out, arg, ref, rarg, dtype == BF16, f"pool {sizes}")
        else:
            check_sum(out, ref, sabs, dtype == BF16, f"pool {sizes}")


def test_validate(pyg):
    ei = to_dev(np.array([[0, 5, -1, 2], [1, 1, 1, 9]], np.int64))
    assert pyg.validate_coo(ei, 6) == 2   # -1 and 9
    assert pyg.validate_coo(ei, 5) == 3   # 5, -1 and 9
    assert pyg.validate_coo(ei, 10) == 1
    assert pyg.validate_batch(to_dev(np.array([0, 0, 1, 1, 3], np.int64)), 4) == 0
    assert pyg.validate_batch(to_dev(np.array([0, 2, 1, 1, 4], np.int64)), 4) == 2


# ------------------------------------------------------ full-size workloads

def test_config1_sparse_uniform(pyg):
    c = synth.make_config(1)
    ei, x, N = c["edge_index"], c["x"], c["N"]
    for kernel in ("coo", "csr"):
        for aggr in ("sum", "mean", "max"):
            run_propagate_case(pyg, ei, x, None, "src", aggr, kernel, what="C1")
    # GCN: gcn_norm-weighted sum with self-loops, the oracle's weights on both sides
    eig = c["edge_index_gcn"]
    w = oracle.gcn_norm(eig, N).astype(np.float32)
    for kernel in ("coo", "csr"):
        run_propagate_case(pyg, eig, x, w, "src", "sum", kernel, what="C1 gcn")
    # and the device chain gcn_norm -> CSR -> propagate against the oracle chain
    d_ei = to_dev(eig)
    norm = pyg.gcn_norm(d_ei, N)
    out, _ = pyg.propagate(to_dev(x), d_ei, norm, csr=pyg.coo_to_csr(d_ei, N, norm), aggr="sum")
    ref, _, sabs = oracle.propagate(x, eig, w, aggr="sum")
    check_sum(out, ref, sabs, what="C1 chain")


@pytest.mark.parametrize("F", [64, 500])
def test_config2_power_law(pyg, F):
    c = synth.make_config(2, F=F)
    N, eig, x = c["N"], c["edge_index_gcn"], c["x"]
    w = oracle.gcn_norm(eig, N).astype(np.float32)
    ei_t = to_dev(eig)
    csr_w = pyg.coo_to_csr(ei_t, N, to_dev(w))
    csr = pyg.coo_to_csr(ei_t, N)
    for kernel in ("coo", "csr"):
        for aggr in ("sum", "mean", "max"):
            run_propagate_case(pyg, eig, x, w, "src", aggr, kernel, csr=csr_w, what=f"C2 F={F} gcn")
        for aggr in ("mean", "max"):
            run_propagate_case(pyg, eig, x, None, "src", aggr, kernel, csr=csr, what=f"C2 F={F}")


def test_config3_minibatch(pyg):
    c = synth.make_config(3)
    N, B, ei, x, batch = c["N"], c["B"], c["edge_index"], c["x"], c["batch"]
    d_ei, d_x, d_b = to_dev(ei), to_dev(x), to_dev(batch)
    csr = pyg.coo_to_csr(d_ei, N)
    for kernel in ("coo", "csr"):
        for aggr in ("sum", "mean", "max"):
            run_propagate_case(pyg, ei, x, None, "src", aggr, kernel, csr=csr, what="C3")
    assert pyg.validate_batch(d_b, B) == 0
    for paggr in ("sum", "mean", "max"):
        # the readout itself on identical inputs: each oracle propagate output, rounded to fp32
        for aggr in ("sum", "mean", "max"):
            h, _, _ = oracle.propagate(x, ei, aggr=aggr)
            h32 = h.astype(np.float32)
            out, arg = pyg.global_pool(to_dev(h32), d_b, B, paggr)
            ref, rarg, sabs = oracle.global_pool(h32, batch, B, paggr)
            if paggr == "max":
                check_max(out, arg, ref, rarg, what=f"C3 pool {aggr}->{paggr}")
            else:
                check_sum(out, ref, sabs, what=f"C3 pool {aggr}->{paggr}")
        # and the device chain propagate(max) -> pool is bit-exact end to end
        hm, _ = pyg.propagate(d_x, csr=csr, aggr="max")
        out, arg = pyg.global_pool(hm, d_b, B, paggr)
        h, _, _ = oracle.propagate(x, ei, aggr="max")
        ref, rarg, sabs = oracle.global_pool(h.astype(np.float32), batch, B, paggr)
        if paggr == "max":
            check_max(out, arg, ref, rarg, what="C3 chain max")
        else:
            check_sum(out, ref, sabs, what=f"C3 chain max->{paggr}")
    # blocks are independent: the packed batch equals per-graph propagates
    out, _ = pyg.propagate(d_x, csr=csr, aggr="sum")
    off = 0
    ends = np.cumsum(c["sizes"])
    for g in (0, 57, 127):
        lo, hi = (ends[g - 1] if g else 0), ends[g]
        m = (ei[1] >= lo) & (ei[1] < hi)
        sub = ei[:, m] - lo
        ref, _, sabs = oracle.propagate(x[lo:hi], sub, aggr="sum")
        check_sum(out[lo:hi], ref, sabs, what=f"C3 block {g}")
    del off


def test_config4_knn(pyg):
    c = synth.make_config(4)
    for key in ("edge_index", "edge_index_shuffled"):
        ei = c[key]
        csr = pyg.coo_to_csr(to_dev(ei), c["N"])
        for kernel in ("coo", "csr"):
            for aggr in ("max", "mean"):
                run_propagate_case(pyg, ei, c["x"], None, "diff", aggr, kernel, csr=csr, what=f"C4 {key}")
