"""Parity at the full size of the large power-law workload (N=232,965,
E~114.8M with self-loops, F=128), in the launch configuration the benchmark
times. Degree, CSR and gcn_norm are compared with the oracle element by
element; propagate on sampled target rows (hubs that span many work chunks
included), whose oracle values are computed from the edges into those rows."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.parity import bf16_round, check_max, check_sum, to_dev

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


@pytest.fixture(scope="module")
def c5():
    c = synth.make_config(5)
    print(f"[c5] generated N={c['N']} E={c['edge_index_gcn'].shape[1]}", flush=True)
    return c


@pytest.fixture(scope="module")
def dev_graph(pyg, c5):
    ei_np = c5["edge_index_gcn"]
    N = c5["N"]
    ei = to_dev(ei_np)
    w_ref = oracle.gcn_norm(ei_np, N).astype(np.float32)
    csr = pyg.coo_to_csr(ei, N, to_dev(w_ref))
    return ei, w_ref, csr


def test_c5_degree_csr_norm_full(pyg, c5, dev_graph):
    ei_np, N = c5["edge_index_gcn"], c5["N"]
    ei, w_ref, csr = dev_graph
    deg_ref = oracle.degree(ei_np, N)
    assert np.array_equal(pyg.degree(ei, N).cpu().numpy(), deg_ref)
    assert np.array_equal(pyg.degree_csr(csr).cpu().numpy(), deg_ref)  # what the benchmark step reports
    rp, col, perm = oracle.coo_to_csr(ei_np, N)
    assert np.array_equal(csr.rowptr.cpu().numpy(), rp)
    assert np.array_equal(csr.perm.cpu().numpy(), perm)
    assert np.array_equal(csr.col.cpu().numpy().astype(np.int64), col)
    del col
    assert np.array_equal(csr.weight.cpu().numpy(), w_ref[perm])
    # unit weights: every fp64 step is order-independent -> identical to the rounded oracle
    assert np.array_equal(pyg.gcn_norm(ei, N).cpu().numpy(), w_ref)
    # the CSR-ordered normalisation the benchmark step uses
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E)
    assert np.array_equal(pyg.gcn_norm_csr(plain).cpu().numpy(), w_ref[perm])


def sample_rows(c5, n=1500):
    ei_np, N = c5["edge_index_gcn"], c5["N"]
    deg = np.bincount(ei_np[1], minlength=N)
    rng = np.random.default_rng(77)
    hubs = np.argsort(deg)[-12:]             # rows split across many chunks
    light = np.argsort(deg, kind="stable")[:12]
    rows = np.unique(np.concatenate([rng.choice(N, n, replace=False), hubs, light]))
    keep = np.isin(ei_np[1], rows)
    return rows, keep


@pytest.mark.parametrize("kernel", ["csr", "coo"])
def test_c5_propagate_sampled(pyg, c5, dev_graph, kernel):
    ei_np, x_np, N = c5["edge_index_gcn"], c5["x"], c5["N"]
    ei, w_ref, csr = dev_graph
    rows, keep = sample_rows(c5)
    sub = ei_np[:, keep]
    kidx = np.nonzero(keep)[0]
    w_sub = w_ref[keep]
    x32 = to_dev(x_np)
    w = to_dev(w_ref)
    cases = [("sum", torch.float32, w), ("mean", torch.float32, w), ("sum", torch.bfloat16, w),
             ("mean", torch.bfloat16, w), ("max", torch.float32, None)]
    for aggr, dt, wt in cases:
        xx = x32.to(dt)
        use = None
        if kernel == "csr":  # the unweighted run reads the same CSR without its weights
            use = csr if wt is not None else pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E)
        out, arg = pyg.propagate(xx, ei, wt, csr=use, aggr=aggr, kernel=kernel)
        torch.cuda.synchronize()
        xin = x_np if dt == torch.float32 else bf16_round(x_np)
        ref, rarg, sabs = oracle.propagate(xin, sub, w_sub if wt is not None else None, aggr=aggr)
        what = f"C5 {kernel} {aggr} {dt}"
        got = out[to_dev(rows)]
        if aggr == "max":
            rarg_full = np.where(rarg[rows] < sub.shape[1], kidx[np.minimum(rarg[rows], sub.shape[1] - 1)],
                                 ei_np.shape[1])
            check_max(got, arg[to_dev(rows)], ref[rows], rarg_full, what=what)
        else:
            check_sum(got, ref[rows], sabs[rows], dt == torch.bfloat16, what)
        print(f"[c5] {what} ok", flush=True)


def test_c5_propagate_backward_sampled(pyg, c5, dev_graph):
    """The gradient of the propagate as the benchmark times it (fp32):
    gcn-weighted sum with the weight gradient, mean, and max through the
    forward's argmax; grad_x on sampled nodes (their outgoing edges in the
    oracle's sub-graph), grad_w on every edge of that sub-graph."""
    ei_np, x_np, N = c5["edge_index_gcn"], c5["x"], c5["N"]
    ei, w_ref, csr = dev_graph
    E = ei_np.shape[1]
    w = to_dev(w_ref)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, w, chunk=csr.chunk)
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, E, csr.chunk)
    plain_t = pyg.CSR(csr_t.rowptr, csr_t.col, csr_t.perm, None, N, E, csr_t.chunk)
    g = np.random.default_rng(81).standard_normal(x_np.shape).astype(np.float32)
    x32, g32 = to_dev(x_np), to_dev(g)
    gx_s, gw_s = pyg.propagate_backward(g32, x32, ei, w, csr=csr, csr_t=csr_t, aggr="sum", need_grad_w=True)
    gx_m, _ = pyg.propagate_backward(g32, x32, ei, None, csr=plain, csr_t=plain_t, aggr="mean")
    torch.cuda.synchronize()
    nodes = sample_rows(c5, n=200)[0]
    keep = np.isin(ei_np[0], nodes)
    kidx = np.nonzero(keep)[0]
    sub = np.ascontiguousarray(ei_np[:, keep])
    # mean divides by the in-degree of each edge's target, taken over the whole graph: the
    # oracle's sub-graph keeps only some of those edges, so mean is checked through s*g
    deg = np.bincount(ei_np[1], minlength=N).astype(np.float64)
    rx, rw, sx, sw = oracle.propagate_backward(x_np, sub, g, w_ref[keep], aggr="sum", want_grad_w=True)
    check_sum(gx_s[to_dev(nodes)].cpu(), rx[nodes], sx[nodes], False, "C5 backward sum grad_x")
    check_sum(gw_s[to_dev(kidx)].cpu(), rw, sw, False, "C5 backward sum grad_w")
    # grad_w in CSR slot order (as the benchmark also times it): the same values at the slots
    _, gw_c = pyg.propagate_backward(g32, x32, ei, w, csr=csr, csr_t=csr_t, aggr="sum", need_grad_w=True,
                                     w_order="csr")
    assert torch.equal(gw_c, gw_s[csr.perm]), "C5 backward sum grad_w in CSR order"
    del gw_c
    gm = (g.astype(np.float64) / np.maximum(deg, 1.0)[:, None]).astype(np.float32)  # rounded like the kernel's s*g
    rxm, _, sxm, _ = oracle.propagate_backward(x_np, sub, gm, aggr="sum")
    check_sum(gx_m[to_dev(nodes)].cpu(), rxm[nodes], sxm[nodes], False, "C5 backward mean grad_x")
    # max: every winner of the sampled target rows; the oracle's own argmax over those rows' edges
    rows, keep_in = sample_rows(c5, n=200)
    sub_in = np.ascontiguousarray(ei_np[:, keep_in])
    kin = np.nonzero(keep_in)[0]
    _, rarg, _ = oracle.propagate(x_np, sub_in, aggr="max")
    arg_full = np.full((N, x_np.shape[1]), E, np.int64)
    arg_full[rows] = np.where(rarg[rows] < sub_in.shape[1], kin[np.minimum(rarg[rows], sub_in.shape[1] - 1)], E)
    gx_x, _ = pyg.propagate_backward(g32, x32, ei, None, csr=plain, csr_t=plain_t, aggr="max",
                                     argmax=to_dev(arg_full))
    torch.cuda.synchronize()
    rxx, _, sxx, _ = oracle.propagate_backward(x_np, ei_np, g, aggr="max", argmax=arg_full)
    check_sum(gx_x.cpu(), rxx, sxx, False, "C5 backward max grad_x")
    print("[c5] propagate backward ok", flush=True)
    del csr_t, gx_s, gw_s, gx_m, gx_x
    torch.cuda.empty_cache()


def test_c5_attention_sampled(pyg, c5, dev_graph):
    """GAT attention at the benchmark's shape (H = 8 heads of 16 columns) in
    CSR slot order: the coefficients of every edge into the sampled rows and
    the attention sum of those rows. A stable CSR keeps each row's edges in
    ascending COO id, so the slots of row r are rowptr[r] + 0, 1, ... over
    np.flatnonzero(target == r)."""
    from tests.parity import check_softmax
    ei_np, x_np, N = c5["edge_index_gcn"], c5["x"], c5["N"]
    _, _, csr = dev_graph
    H = 8
    rng = np.random.default_rng(78)
    a_src = rng.standard_normal((N, H)).astype(np.float32)
    a_dst = rng.standard_normal((N, H)).astype(np.float32)
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E)
    alpha = pyg.gat_softmax(to_dev(a_src), to_dev(a_dst), plain, 0.2, "csr")
    out = pyg.propagate_heads(to_dev(x_np), plain, alpha, H)
    torch.cuda.synchronize()
    rows, keep = sample_rows(c5, n=400)
    sub = np.ascontiguousarray(ei_np[:, keep])
    rowptr = np.concatenate([[0], np.cumsum(np.bincount(ei_np[1], minlength=N))])
    order = np.argsort(sub[1], kind="stable")  # sub edges grouped by row, ascending id inside a row
    dst_sorted = sub[1][order]
    first = np.searchsorted(dst_sorted, dst_sorted)  # first position of each row's run
    slots = rowptr[dst_sorted] + (np.arange(order.size) - first)
    got = alpha[to_dev(slots)].cpu()
    e = oracle.gat_scores(a_src, a_dst, sub, 0.2)
    ref = oracle.segment_softmax(e, sub, N)
    check_softmax(got, ref[order], e[order], dst_sorted, N, "C5 gat_softmax")
    ref_out, sabs = oracle.propagate_heads(x_np, sub, ref.astype(np.float32), H)
    g = out[to_dev(rows)].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(g - ref_out[rows]) <= 2e-5 * sabs[rows] + 1e-6), "C5 propagate_heads"
    # the attention sum in bf16 storage with the GPU's coefficients' own oracle (alpha from the oracle, fp32)
    alpha_ref = torch.zeros(csr.E, H)
    alpha_ref[torch.from_numpy(slots)] = torch.from_numpy(ref[order].astype(np.float32))
    outb = pyg.propagate_heads(to_dev(x_np).to(torch.bfloat16), plain, alpha_ref.to("cuda"), H)
    torch.cuda.synchronize()
    ref_b, sabs_b = oracle.propagate_heads(bf16_round(x_np), sub, ref.astype(np.float32), H)
    check_sum(outb[to_dev(rows)].cpu(), ref_b[rows], sabs_b[rows], True, "C5 propagate_heads bf16")
    print("[c5] attention ok", flush=True)


def test_c5_softmax_scores_sampled(pyg, c5, dev_graph):
    """The softmax of given scores and its backward at the benchmark's shape
    (H = 8, CSR slot order): every edge into the sampled rows. Scores,
    coefficients and upstream gradients from the counter-based generator
    (row k = COO edge k)."""
    from synth.hashed import hashed_matrix, hashed_values
    from tests.parity import check_softmax
    ei_np, N = c5["edge_index_gcn"], c5["N"]
    _, _, csr = dev_graph
    E, H = ei_np.shape[1], 8
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E)
    d_perm = csr.perm
    sc = hashed_matrix(E, H, seed=31, device="cuda")[d_perm] * 4.0
    al = hashed_matrix(E, H, seed=37, device="cuda")[d_perm] * 0.5 + 0.5
    gg = hashed_matrix(E, H, seed=41, device="cuda")[d_perm]
    alpha = pyg.segment_softmax(sc, plain, "csr")
    gsc = pyg.segment_softmax_backward(al, gg, plain, "csr")
    torch.cuda.synchronize()
    del sc, al, gg
    rows, keep = sample_rows(c5, n=400)
    kidx = np.nonzero(keep)[0]
    sub = np.ascontiguousarray(ei_np[:, keep])
    rowptr = np.concatenate([[0], np.cumsum(np.bincount(ei_np[1], minlength=N))])
    order = np.argsort(sub[1], kind="stable")
    dst_sorted = sub[1][order]
    first = np.searchsorted(dst_sorted, dst_sorted)
    slots = rowptr[dst_sorted] + (np.arange(order.size) - first)
    s_sub = hashed_values(torch.from_numpy(kidx), H, seed=31).numpy() * np.float32(4.0)
    ref = oracle.segment_softmax(s_sub, sub, N)
    check_softmax(alpha[to_dev(slots)].cpu(), ref[order], s_sub[order], dst_sorted, N, "C5 segment_softmax")
    a_sub = hashed_values(torch.from_numpy(kidx), H, seed=37).numpy() * np.float32(0.5) + np.float32(0.5)
    g_sub = hashed_values(torch.from_numpy(kidx), H, seed=41).numpy()
    rb, sabs = oracle.segment_softmax_backward(a_sub, g_sub, sub, N)
    err = np.abs(gsc[to_dev(slots)].cpu().numpy().astype(np.float64) - rb[order])
    assert np.all(err <= 1e-5 * sabs[order] + 1e-12), f"C5 softmax backward: {np.max(err / (1e-5 * sabs[order] + 1e-12))}"
    print("[c5] softmax of scores and backward ok", flush=True)
    del alpha, gsc
    torch.cuda.empty_cache()


def test_c5_whole_graph_pool(pyg, c5):
    """The benchmark's readout shape: one graph of all 232,965 nodes, F = 128,
    mean (also sum and max), over the graph's features."""
    x_np, N = c5["x"], c5["N"]
    batch = np.zeros(N, dtype=np.int64)
    for aggr in ("mean", "sum", "max"):
        out, arg = pyg.global_pool(to_dev(x_np), to_dev(batch), 1, aggr)
        torch.cuda.synchronize()
        ref, rarg, sabs = oracle.global_pool(x_np, batch, 1, aggr)
        if aggr == "max":
            check_max(out, arg, ref, rarg, what="C5 pool max")
        else:
            check_sum(out, ref, sabs, False, f"C5 pool {aggr}")
    print("[c5] whole-graph pool ok", flush=True)


def test_c5_attention_backward_sampled(pyg, c5, dev_graph):
    """The attention backward at the benchmark's shape (H = 8 heads of 16
    columns, fp32, coefficients and score gradients in CSR slot order, the
    reversed CSR and the transpose map as the benchmark builds them). The
    transpose map is compared in full with the one the oracle's two CSR
    permutations define; the gradients on sampled nodes (their whole
    neighbourhoods taken into the oracle's sub-graph) and on every edge of
    that sub-graph. Coefficients and score gradients come from the
    counter-based generator, so that the oracle can regenerate the rows of
    its sub-graph."""
    from synth.hashed import hashed_matrix, hashed_values
    ei_np, x_np, N = c5["edge_index_gcn"], c5["x"], c5["N"]
    ei, _, csr = dev_graph
    E, F, H = ei_np.shape[1], x_np.shape[1], 8
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, chunk=csr.chunk)
    map_t = pyg.csr_transpose_map(plain, csr_t)
    _, _, perm = oracle.coo_to_csr(ei_np, N)
    _, _, perm_t = oracle.coo_to_csr(np.ascontiguousarray(ei_np[::-1]), N)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(E)
    assert np.array_equal(map_t.cpu().numpy().astype(np.int64), inv[perm_t]), "C5 transpose map"
    del perm_t
    print("[c5] transpose map ok", flush=True)

    rng = np.random.default_rng(79)
    g = rng.standard_normal((N, F)).astype(np.float32)
    a_src = rng.standard_normal((N, H)).astype(np.float32)
    a_dst = rng.standard_normal((N, H)).astype(np.float32)
    d_perm = to_dev(perm)
    alpha = hashed_matrix(E, H, seed=23, device="cuda")[d_perm]   # row k of the generator = COO edge k
    gsc = hashed_matrix(E, H, seed=29, device="cuda")[d_perm]
    gx, galpha = pyg.propagate_heads_backward(to_dev(g), to_dev(x_np), plain, csr_t, alpha, H, map_t=map_t)
    gxb, galphab = pyg.propagate_heads_backward(to_dev(g).to(torch.bfloat16), to_dev(x_np).to(torch.bfloat16), plain,
                                                csr_t, alpha, H, map_t=map_t)
    gs, gd = pyg.gat_scores_backward(to_dev(a_src), to_dev(a_dst), plain, csr_t, gsc, 0.2, map_t=map_t)
    torch.cuda.synchronize()
    del alpha, gsc
    nodes = sample_rows(c5, n=300)[0]
    keep = np.isin(ei_np[0], nodes) | np.isin(ei_np[1], nodes)  # whole out- and in-neighbourhoods
    kidx = np.nonzero(keep)[0]
    sub = np.ascontiguousarray(ei_np[:, keep])
    al_sub = hashed_values(torch.from_numpy(kidx), H, seed=23).numpy()
    gs_sub = hashed_values(torch.from_numpy(kidx), H, seed=29).numpy()
    rx, ra, sx, sa = oracle.propagate_heads_backward(x_np, sub, al_sub, g, H)
    check_sum(gx[to_dev(nodes)].cpu(), rx[nodes], sx[nodes], False, "C5 attention backward grad_x")
    slots = inv[kidx]
    check_sum(galpha[to_dev(slots)].cpu(), ra, sa, False, "C5 attention backward grad_alpha")
    rxb, rab, sxb, sab = oracle.propagate_heads_backward(bf16_round(x_np), sub, al_sub, bf16_round(g), H)
    check_sum(gxb[to_dev(nodes)].cpu(), rxb[nodes], sxb[nodes], True, "C5 attention backward grad_x bf16")
    check_sum(galphab[to_dev(slots)].cpu(), rab, sab, False, "C5 attention backward grad_alpha bf16 inputs")
    rs, rd, ss, sd = oracle.gat_scores_backward(a_src, a_dst, sub, gs_sub, 0.2)
    check_sum(gs[to_dev(nodes)].cpu(), rs[nodes], ss[nodes], False, "C5 score backward grad_a_src")
    check_sum(gd[to_dev(nodes)].cpu(), rd[nodes], sd[nodes], False, "C5 score backward grad_a_dst")
    print("[c5] attention backward ok", flush=True)
    del csr_t, map_t, gx, galpha, gxb, galphab
    torch.cuda.empty_cache()


def test_c5_edge_features_sampled(pyg, c5, dev_graph):
    """Edge-feature messages at the benchmark's shape: every edge of the large
    graph carries a 128-dimensional feature (counter-based, regenerable for
    any subset of edges); max(x_j + e, 0) with sum (the benchmark's call, fp32
    and bf16, features in CSR slot order) plus the other two messages with
    mean and max (features in COO order), checked on sampled target rows."""
    from synth.hashed import hashed_matrix, hashed_values
    ei_np, x_np, N = c5["edge_index_gcn"], c5["x"], c5["N"]
    ei, _, csr = dev_graph
    E, F = ei_np.shape[1], x_np.shape[1]
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E)
    ea = hashed_matrix(E, F, seed=17, device="cuda")
    ea_csr = ea[csr.perm]  # rows in CSR slot order, as the benchmark passes them
    rows, keep = sample_rows(c5, n=300)
    sub = np.ascontiguousarray(ei_np[:, keep])
    kidx = np.nonzero(keep)[0]
    ea_sub = hashed_values(torch.from_numpy(kidx), F, seed=17).numpy()
    x32 = to_dev(x_np)
    cases = [("edge_relu", "sum", torch.float32, "csr"), ("edge_relu", "sum", torch.bfloat16, "csr"),
             ("edge_add", "mean", torch.float32, "coo"), ("edge_mul", "max", torch.float32, "coo")]
    for msg, aggr, dt, order in cases:
        feats = (ea_csr if order == "csr" else ea).to(dt)
        out, arg = pyg.propagate_edge(x32.to(dt), feats, ei, plain, msg, aggr, "csr", order)
        torch.cuda.synchronize()
        bf = dt == torch.bfloat16
        xin = bf16_round(x_np) if bf else x_np
        ein = bf16_round(ea_sub) if bf else ea_sub
        ref, rarg, sabs = oracle.propagate(xin, sub, msg=msg, aggr=aggr, edge_attr=ein)
        what = f"C5 edge {msg} {aggr} {dt} {order}"
        got = out[to_dev(rows)]
        if aggr == "max":
            rarg_full = np.where(rarg[rows] < sub.shape[1], kidx[np.minimum(rarg[rows], sub.shape[1] - 1)], E)
            check_max(got, arg[to_dev(rows)], ref[rows], rarg_full, what=what)
        else:
            check_sum(got, ref[rows], sabs[rows], bf, what)
        print(f"[c5] {what} ok", flush=True)
        del feats
    del ea, ea_csr
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_c5_edge_backward_sampled(pyg, c5, dev_graph, dtype):
    """The backward of the benchmark's edge-feature call (max(x_j + e, 0),
    sum, features in CSR slot order, fp32 and bf16): grad_x on sampled nodes
    (all their outgoing edges in the oracle's sub-graph) and grad_e on every
    edge of that sub-graph. bf16: the oracle sees the bf16-rounded values."""
    from synth.hashed import hashed_matrix, hashed_values
    bf16 = dtype == torch.bfloat16
    ei_np, x_np, N = c5["edge_index_gcn"], c5["x"], c5["N"]
    ei, _, csr = dev_graph
    E, F = ei_np.shape[1], x_np.shape[1]
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E)
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, chunk=csr.chunk)
    map_t = pyg.csr_transpose_map(plain, csr_t)
    ea_csr = hashed_matrix(E, F, seed=43, device="cuda")[csr.perm].to(dtype)  # row k of the generator = COO edge k
    g = np.random.default_rng(80).standard_normal((N, F)).astype(np.float32)
    xs = x_np
    if bf16:
        g, xs = bf16_round(g), bf16_round(x_np)
    gx, ge = pyg.propagate_edge_backward(to_dev(g).to(dtype), to_dev(xs).to(dtype), ea_csr, plain, "edge_relu", "sum",
                                         "csr", csr_t=csr_t, map_t=map_t)
    torch.cuda.synchronize()
    del ea_csr
    nodes = sample_rows(c5, n=200)[0]
    keep = np.isin(ei_np[0], nodes)
    kidx = np.nonzero(keep)[0]
    sub = np.ascontiguousarray(ei_np[:, keep])
    ea_sub = hashed_values(torch.from_numpy(kidx), F, seed=43).numpy()
    if bf16:
        ea_sub = bf16_round(ea_sub)
    rx, re, sx, se = oracle.propagate_edge_backward(xs, sub, ea_sub, g, "edge_relu", "sum")
    check_sum(gx[to_dev(nodes)].cpu(), rx[nodes], sx[nodes], bf16, f"C5 edge backward {dtype} grad_x")
    _, _, perm = oracle.coo_to_csr(ei_np, N)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(E)
    check_sum(ge[to_dev(inv[kidx])].cpu(), re, se, bf16, f"C5 edge backward {dtype} grad_e")
    print(f"[c5] edge backward {dtype} ok", flush=True)
    del gx, ge, csr_t, map_t
    torch.cuda.empty_cache()


def test_c5_dense_transform_sampled(pyg, c5):
    """The matrix-core X Theta at the benchmark's shape (N=232,965, 128 -> 128,
    bf16 operands, bf16 and fp32 out), sampled rows against the oracle."""
    x_np = c5["x"]
    rng = np.random.default_rng(79)
    xb = bf16_round(x_np)
    t = bf16_round((rng.standard_normal((128, 128)) / np.sqrt(128)).astype(np.float32))
    rows = np.sort(rng.choice(x_np.shape[0], 2000, replace=False))
    ref, sabs = oracle.dense_transform(xb[rows], t)
    for odt in (torch.bfloat16, torch.float32):
        out = pyg.dense_transform(to_dev(xb).to(torch.bfloat16), to_dev(t).to(torch.bfloat16), odt)
        torch.cuda.synchronize()
        check_sum(out[to_dev(rows)], ref, sabs, odt == torch.bfloat16, f"C5 dense {odt}")
    # fp32 operands (the fp32 matrix-core path) on the benchmark's fp32 features
    t32 = (rng.standard_normal((128, 128)) / np.sqrt(128)).astype(np.float32)
    ref32, sabs32 = oracle.dense_transform(x_np[rows], t32)
    out = pyg.dense_transform(to_dev(x_np), to_dev(t32), torch.float32)
    torch.cuda.synchronize()
    check_sum(out[to_dev(rows)], ref32, sabs32, False, "C5 dense fp32 operands")


@pytest.fixture(scope="module")
def c5_oracle_full(c5):
    """The oracle over the whole large graph (every row): the gcn-weighted sum
    and mean of fp32 x, the sum of the bf16-rounded x, and the unweighted max
    with argmax. Four independent single-threaded oracle calls, run side by
    side (each releases the interpreter while it loops)."""
    import concurrent.futures as cf
    ei_np, x_np, N = c5["edge_index_gcn"], c5["x"], c5["N"]
    w_ref = oracle.gcn_norm(ei_np, N).astype(np.float32)
    xb = bf16_round(x_np)
    jobs = {"sum": (x_np, w_ref, "sum"), "mean": (x_np, w_ref, "mean"), "sum_bf16": (xb, w_ref, "sum"),
            "max": (x_np, None, "max")}
    with cf.ThreadPoolExecutor(len(jobs)) as ex:
        futs = {k: ex.submit(oracle.propagate, xx, ei_np, ww, aggr=a) for k, (xx, ww, a) in jobs.items()}
        res = {k: f.result() for k, f in futs.items()}
    print("[c5] full-graph oracle done", flush=True)
    return res


def test_c5_propagate_every_row(pyg, c5, dev_graph, c5_oracle_full):
    """The benchmark's propagate (gcn-weighted sum, CSR kernel, the launch
    configuration it times) on every row of the large graph, and the same
    CSR with mean, bf16 rows and max / argmax (bit for bit), against the
    oracle's whole-graph results."""
    x_np, N = c5["x"], c5["N"]
    ei, w_ref, csr = dev_graph
    x32 = to_dev(x_np)
    ref = c5_oracle_full
    out, _ = pyg.propagate(x32, csr=csr, aggr="sum")
    torch.cuda.synchronize()
    r = check_sum(out, ref["sum"][0], ref["sum"][2], False, "C5 every row: fp32 gcn-weighted sum (CSR)")
    print(f"[c5] every row fp32 sum ok (worst error / bound {r:.3f})", flush=True)
    out, _ = pyg.propagate(x32, csr=csr, aggr="mean")
    torch.cuda.synchronize()
    check_sum(out, ref["mean"][0], ref["mean"][2], False, "C5 every row: fp32 gcn-weighted mean (CSR)")
    out, _ = pyg.propagate(x32.to(torch.bfloat16), csr=csr, aggr="sum")
    torch.cuda.synchronize()
    check_sum(out, ref["sum_bf16"][0], ref["sum_bf16"][2], True, "C5 every row: bf16 gcn-weighted sum (CSR)")
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E, csr.chunk)
    out, arg = pyg.propagate(x32, csr=plain, aggr="max")
    torch.cuda.synchronize()
    check_max(out, arg, ref["max"][0], ref["max"][1], what="C5 every row: fp32 max / argmax (CSR)")
    print("[c5] every row: sum, mean, bf16 sum, max ok", flush=True)


@pytest.mark.parametrize("B", [2, 8])
def test_c5_propagate_blocked_every_row(pyg, c5, dev_graph, c5_oracle_full, B):
    """The source-blocked propagate on every row of the large graph: the
    gcn-weighted sum in fp32 and bf16, and max / argmax bit for bit."""
    x_np, N = c5["x"], c5["N"]
    ei, w_ref, csr = dev_graph
    ref = c5_oracle_full
    x32 = to_dev(x_np)
    bc = pyg.csr_blocks(csr, B)
    out, _ = pyg.propagate_blocked(x32, bc, "sum")
    torch.cuda.synchronize()
    check_sum(out, ref["sum"][0], ref["sum"][2], False, f"C5 every row: blocked B={B} fp32 sum")
    out, _ = pyg.propagate_blocked(x32.to(torch.bfloat16), bc, "sum")
    torch.cuda.synchronize()
    check_sum(out, ref["sum_bf16"][0], ref["sum_bf16"][2], True, f"C5 every row: blocked B={B} bf16 sum")
    del bc
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E, csr.chunk)
    bp = pyg.csr_blocks(plain, B, with_perm=True)
    out, arg = pyg.propagate_blocked(x32, bp, "max")
    torch.cuda.synchronize()
    check_max(out, arg, ref["max"][0], ref["max"][1], what=f"C5 every row: blocked B={B} max / argmax")
    print(f"[c5] every row: blocked B={B} ok", flush=True)


def test_c5_gcn_propagate_every_row(pyg, c5, dev_graph, c5_oracle_full):
    """The fused GCN propagate (the benchmark step's call) on the large graph:
    norms bit for bit against the oracle's, every output row against the
    oracle's gcn-weighted sum."""
    x_np, N = c5["x"], c5["N"]
    ei, w_ref, csr = dev_graph
    plain = pyg.CSR(csr.rowptr, csr.col, csr.perm, None, N, csr.E, csr.chunk)
    norm = torch.empty(csr.E, device="cuda")
    out = pyg.gcn_propagate(to_dev(x_np), plain, norm_out=norm)
    torch.cuda.synchronize()
    assert torch.equal(norm, csr.weight), "C5 fused norms differ from the oracle's (in CSR order)"
    r = check_sum(out, c5_oracle_full["sum"][0], c5_oracle_full["sum"][2], False, "C5 every row: fused GCN propagate")
    print(f"[c5] every row: fused GCN propagate ok (worst error / bound {r:.3f})", flush=True)


def test_c5_gcn_propagate_blocked_every_row(pyg, c5, dev_graph, c5_oracle_full):
    """The fused GCN propagate over the two-block source-blocked CSR (the
    benchmark step's call): norms bit for bit against the oracle's (carried
    into the blocked slot order), every output row against the oracle's
    gcn-weighted sum, fp32 and bf16."""
    x_np, N = c5["x"], c5["N"]
    ei, w_ref, csr = dev_graph
    # the step's calls: the blocked CSR straight from the COO, d from it
    bplain = pyg.coo_to_csr_blocked(ei, N, 2)
    deg = pyg.degree_csr_blocks(bplain)
    norm = torch.empty(csr.E, device="cuda")
    out = pyg.gcn_propagate_blocked(to_dev(x_np), None, bplain, norm_out=norm)
    ref_b = pyg.csr_blocks(csr, 2)  # the oracle's norms in the blocked slot order
    torch.cuda.synchronize()
    assert torch.equal(bplain.rowptr, ref_b.rowptr) and torch.equal(bplain.col, ref_b.col), \
        "C5 blocked CSR from the COO differs from the regrouped CSR"
    assert np.array_equal(deg.cpu().numpy(), oracle.degree(c5["edge_index_gcn"], N))
    ref_norm = ref_b.weight
    del ref_b
    assert torch.equal(norm, ref_norm), "C5 blocked fused norms differ from the oracle's"
    r = check_sum(out, c5_oracle_full["sum"][0], c5_oracle_full["sum"][2], False,
                  "C5 every row: blocked fused GCN propagate")
    del ref_norm
    # without norms (the benchmark step's call): every window pre-scaled
    out = pyg.gcn_propagate_blocked(to_dev(x_np), None, bplain)
    torch.cuda.synchronize()
    r2 = check_sum(out, c5_oracle_full["sum"][0], c5_oracle_full["sum"][2], False,
                   "C5 every row: blocked GCN propagate, rows pre-scaled")
    print(f"[c5] every row: blocked GCN propagate without norms ok (worst error / bound {r2:.3f})", flush=True)
    outb = pyg.gcn_propagate_blocked(to_dev(x_np).to(torch.bfloat16), None, bplain)
    torch.cuda.synchronize()
    check_sum(outb, c5_oracle_full["sum_bf16"][0], c5_oracle_full["sum_bf16"][2], True,
              "C5 every row: blocked fused GCN propagate bf16")
    print(f"[c5] every row: blocked fused GCN propagate ok (worst error / bound {r:.3f})", flush=True)
