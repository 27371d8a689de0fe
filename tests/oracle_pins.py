"""Pins that tie the oracle to something other than itself.

Each pin checks the oracle against an independent source: hand-derived
values (tests/golden/tiny_hand.json), dense linear algebra in numpy,
CPU torch scatter routines, closed forms and invariants of Eq. (1).
Every pin is a function of the oracle library handle, so the mutation test
can run the same pins against deliberately broken copies of the oracle.
"""
from __future__ import annotations

import json
import os

import numpy as np
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "tiny_hand.json")


def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def dense_adjacency(ei, N, w=None):
    """A[i, j] = sum of weights of edges j -> i (dense fp64)."""
    A = np.zeros((N, N))
    np.add.at(A, (ei[1], ei[0]), 1.0 if w is None else np.asarray(w, np.float64))
    return A


def circulant(N, half_k):
    """k-regular symmetric graph (k = 2 half_k): i -> i +- 1..half_k mod N."""
    src, dst = [], []
    for i in range(N):
        for s in range(1, half_k + 1):
            for j in ((i + s) % N, (i - s) % N):
                src.append(j)
                dst.append(i)
    return np.array([src, dst], np.int64)


def small_cases():
    """Tiny random multigraphs with duplicates, self-loops and isolated nodes."""
    rng = np.random.default_rng(1234)
    cases = []
    for N, E, dup in ((1, 0, True), (1, 3, True), (5, 0, True), (7, 20, True), (16, 60, True), (33, 200, True),
                      (64, 90, True), (40, 300, False), (90, 700, False)):
        F = int(rng.integers(1, 6))
        ei = synth.random_coo(rng, N, E, duplicates=dup)
        E = ei.shape[1]
        x = rng.standard_normal((N, F)).astype(np.float32)
        w = rng.standard_normal(E).astype(np.float32)
        cases.append((N, F, ei, x, w))
    return cases


# ----------------------------------------------------------------- pins

def pin_golden_propagate(lib):
    g = golden()["propagate"]
    x = np.array(g["x"], np.float32)
    ei = np.array(g["edge_index"], np.int64)
    w = np.array(g["edge_weight"], np.float32)
    N = g["N"]
    assert (oracle.degree(ei, N, lib=lib) == np.array(g["degree"])).all()
    rp, col, perm = oracle.coo_to_csr(ei, N, lib=lib)
    assert (rp == g["csr_rowptr"]).all() and (col == g["csr_col"]).all() and (perm == g["csr_perm"]).all()
    out, _, _ = oracle.propagate(x, ei, aggr="sum", lib=lib)
    assert np.array_equal(out, np.array(g["src_sum"]))
    out, _, _ = oracle.propagate(x, ei, aggr="mean", lib=lib)
    assert np.allclose(out * 3.0, np.array(g["src_mean_times_3"]), rtol=1e-15, atol=0)
    out, arg, _ = oracle.propagate(x, ei, aggr="max", lib=lib)
    assert np.array_equal(out, np.array(g["src_max"])) and np.array_equal(arg, np.array(g["src_argmax"]))
    out, _, _ = oracle.propagate(x, ei, w, aggr="sum", lib=lib)
    assert np.array_equal(out, np.array(g["weighted_sum"]))
    out, arg, _ = oracle.propagate(x, ei, w, aggr="max", lib=lib)
    assert np.array_equal(out, np.array(g["weighted_max"])) and np.array_equal(arg, np.array(g["weighted_argmax"]))
    out, _, _ = oracle.propagate(x, ei, msg="diff", aggr="sum", lib=lib)
    assert np.array_equal(out, np.array(g["diff_sum"]))
    out, arg, _ = oracle.propagate(x, ei, msg="diff", aggr="max", lib=lib)
    assert np.array_equal(out, np.array(g["diff_max"])) and np.array_equal(arg, np.array(g["diff_argmax"]))


def pin_golden_pool(lib):
    g = golden()
    x = np.array(g["propagate"]["x"], np.float32)
    p = g["pool"]
    batch = np.array(p["batch"], np.int64)
    for aggr in ("sum", "mean", "max"):
        out, arg, _ = oracle.global_pool(x, batch, p["B"], aggr, lib=lib)
        assert np.array_equal(out, np.array(p[aggr])), aggr
        if aggr == "max":
            assert np.array_equal(arg, np.array(p["argmax"]))


def pin_golden_gcn_norm(lib):
    g = golden()["gcn_norm_path3"]
    ei = np.array(g["edge_index"], np.int64)
    norm = oracle.gcn_norm(ei, g["N"], lib=lib)
    assert np.allclose(norm * norm, g["norm_squared"], rtol=1e-14, atol=0)
    assert np.allclose(norm, g["norm"], rtol=1e-14, atol=0)


def pin_golden_gcn_norm_directed(lib):
    g = golden()["gcn_norm_directed"]
    ei = np.array(g["edge_index"], np.int64)
    norm = oracle.gcn_norm(ei, g["N"], lib=lib)
    assert np.allclose(norm * norm, g["norm_squared"], rtol=1e-14, atol=0)
    assert np.array_equal(oracle.degree(ei, g["N"], lib=lib), g["degree_with_loops"])


def pin_golden_signed_zero(lib):
    g = golden()["signed_zero_max"]
    x = np.array(g["x"], np.float32)
    ei = np.array(g["edge_index"], np.int64)
    out, arg, _ = oracle.propagate(x, ei, aggr="max", lib=lib)
    assert np.array_equal(out, np.array(g["max"])) and np.array_equal(arg, np.array(g["argmax"]))
    assert not np.signbit(out[2, 0])


def pin_degree_and_csr_library(lib):
    """np.bincount and a stable argsort are independent definitions."""
    for N, F, ei, x, w in small_cases():
        deg = oracle.degree(ei, N, lib=lib)
        assert np.array_equal(deg, np.bincount(ei[1], minlength=N))
        assert deg.sum() == ei.shape[1]
        rp, col, perm = oracle.coo_to_csr(ei, N, lib=lib)
        ref_perm = np.argsort(ei[1], kind="stable")
        assert np.array_equal(perm, ref_perm)
        assert np.array_equal(col, ei[0][ref_perm])
        assert np.array_equal(rp, np.concatenate([[0], np.cumsum(np.bincount(ei[1], minlength=N))]))


def pin_sum_mean_dense(lib):
    """Sum = dense A @ X (fp64 matmul); mean = D^-1 A X; weighted and diff forms."""
    for N, F, ei, x, w in small_cases():
        x64 = x.astype(np.float64)
        deg = np.bincount(ei[1], minlength=N).astype(np.float64)
        for weighted in (False, True):
            A = dense_adjacency(ei, N, w if weighted else None)
            ref = A @ x64
            out, _, sabs = oracle.propagate(x, ei, w if weighted else None, aggr="sum", lib=lib)
            assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)
            Aabs = dense_adjacency(ei, N, np.abs(w) if weighted else None)
            assert np.allclose(sabs, Aabs @ np.abs(x64), rtol=1e-12, atol=1e-12)
            out, _, _ = oracle.propagate(x, ei, w if weighted else None, aggr="mean", lib=lib)
            ref_mean = np.where(deg[:, None] > 0, ref / np.maximum(deg, 1)[:, None], 0.0)
            assert np.allclose(out, ref_mean, rtol=1e-12, atol=1e-12)
        # diff: sum_j (x_j - x_i) = A x - deg * x_i
        A = dense_adjacency(ei, N)
        out, _, _ = oracle.propagate(x, ei, msg="diff", aggr="sum", lib=lib)
        assert np.allclose(out, A @ x64 - deg[:, None] * x64, rtol=1e-12, atol=1e-12)


def pin_torch_scatter(lib):
    """CPU torch index_add_ / scatter_reduce give sum, mean and amax."""
    for N, F, ei, x, w in small_cases():
        E = ei.shape[1]
        xt = torch.from_numpy(x.astype(np.float64))
        msg = xt[torch.from_numpy(ei[0])] * torch.from_numpy(w.astype(np.float64))[:, None]
        idx = torch.from_numpy(ei[1])
        ref = torch.zeros(N, F, dtype=torch.float64).index_add_(0, idx, msg).numpy()
        out, _, _ = oracle.propagate(x, ei, w, aggr="sum", lib=lib)
        assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)
        ref = torch.zeros(N, F, dtype=torch.float64).scatter_reduce(
            0, idx[:, None].expand(E, F), msg, "mean", include_self=False).numpy()
        out, _, _ = oracle.propagate(x, ei, w, aggr="mean", lib=lib)
        assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)
        m32 = torch.from_numpy(x)[torch.from_numpy(ei[0])]
        ref = torch.zeros(N, F, dtype=torch.float32).scatter_reduce(
            0, idx[:, None].expand(E, F), m32, "amax", include_self=False).numpy()
        out, _, _ = oracle.propagate(x, ei, aggr="max", lib=lib)
        assert np.array_equal(out.astype(np.float32), ref)


def pin_max_bruteforce(lib):
    """Max/argmax by scanning a masked message tensor; lowest edge id wins ties."""
    rng = np.random.default_rng(99)
    for N, F, ei, x, w in small_cases():
        # quantise features so that exact ties occur often
        xq = np.round(x * 2).astype(np.float32) * np.float32(0.5)
        E = ei.shape[1]
        for kind in ("src", "weighted", "diff"):
            if kind == "src":
                m = xq[ei[0]]
            elif kind == "weighted":
                wq = np.round(w * 2).astype(np.float32) * np.float32(0.5)
                m = (wq[:, None] * xq[ei[0]]).astype(np.float32)
            else:
                m = (xq[ei[0]] - xq[ei[1]]).astype(np.float32)
            m = np.where(m == 0, np.float32(0), m)
            ref = np.zeros((N, F), np.float32)
            ref_arg = np.full((N, F), E, np.int64)
            for i in range(N):
                ks = np.nonzero(ei[1] == i)[0]
                if ks.size:
                    sub = m[ks]
                    ref[i] = sub.max(axis=0)
                    ref_arg[i] = ks[np.argmax(sub == ref[i][None, :], axis=0)]
            out, arg, _ = oracle.propagate(
                xq, ei, wq if kind == "weighted" else None,
                msg="diff" if kind == "diff" else "src", aggr="max", lib=lib)
            assert np.array_equal(out.astype(np.float32), ref), kind
            assert np.array_equal(arg, ref_arg), kind
            has = arg < E
            if has.any():
                fidx = np.broadcast_to(np.arange(F), arg.shape)
                assert np.array_equal(m[arg[has], fidx[has]], out.astype(np.float32)[has])
    del rng


def pin_gcn_norm_closed_forms(lib):
    """k-regular + self-loops gives 1/(k+1); symmetry; dense D^-1/2 (A) D^-1/2;
    and the eigen-identity  A_hat sqrt(d) = sqrt(d)."""
    for N, hk in ((5, 1), (12, 2), (40, 3)):
        ei = synth.with_self_loops(circulant(N, hk), N)
        norm = oracle.gcn_norm(ei, N, lib=lib)
        assert np.allclose(norm, 1.0 / (2 * hk + 1), rtol=1e-15, atol=0)
    rng = np.random.default_rng(7)
    for N, M in ((6, 5), (30, 60), (80, 200)):
        pairs = synth.uniform_pairs(N, M, rng)
        ei = synth.with_self_loops(synth.symmetrize(pairs), N)
        for weighted in (False, True):
            w = rng.uniform(0.5, 2.0, M) if weighted else None
            wfull = None if w is None else np.concatenate([w, w, np.ones(N)])
            norm = oracle.gcn_norm(ei, N, wfull, lib=lib)
            A = dense_adjacency(ei, N, wfull)
            d = A.sum(axis=1)
            Dm = np.diag(1.0 / np.sqrt(d))
            Ahat = Dm @ A @ Dm
            ref = Ahat[ei[1], ei[0]] / A[ei[1], ei[0]] * (1.0 if wfull is None else wfull)
            assert np.allclose(norm, ref, rtol=1e-13, atol=0)
            # symmetry: edge u->v and v->u share the norm
            E2 = 2 * M
            assert np.allclose(norm[:M], norm[M:E2], rtol=1e-15, atol=0)
            # eigen-identity through the oracle's own propagate
            x = np.repeat(np.sqrt(d)[:, None], 3, axis=1).astype(np.float32)
            out, _, sabs = oracle.propagate(x, ei, norm.astype(np.float32), aggr="sum", lib=lib)
            assert np.allclose(out, np.sqrt(d)[:, None], rtol=2e-6, atol=0)
    # isolated node (no self-loop) -> its outgoing edges get norm 0
    ei = np.array([[0, 1], [1, 1]], np.int64)
    norm = oracle.gcn_norm(ei, 3, lib=lib)
    assert norm[0] == 0.0 and abs(norm[1] - 0.5) <= 1e-15


def pin_invariants(lib):
    """Permutation invariance, sum = mean * deg, isolated nodes, block-diagonal
    batching (no messages between disconnected graphs) and the DIFF identity."""
    rng = np.random.default_rng(5)
    for N, F, ei, x, w in small_cases():
        E = ei.shape[1]
        p = rng.permutation(E)
        eip, wp = ei[:, p], w[p]
        s1, _, _ = oracle.propagate(x, ei, w, aggr="sum", lib=lib)
        s2, _, _ = oracle.propagate(x, eip, wp, aggr="sum", lib=lib)
        assert np.allclose(s1, s2, rtol=1e-12, atol=1e-12)
        m1, _, _ = oracle.propagate(x, ei, w, aggr="mean", lib=lib)
        deg = np.bincount(ei[1], minlength=N)
        assert np.allclose(m1 * deg[:, None], s1, rtol=1e-12, atol=1e-12)
        mx1, a1, _ = oracle.propagate(x, ei, w, aggr="max", lib=lib)
        mx2, a2, _ = oracle.propagate(x, eip, wp, aggr="max", lib=lib)
        assert np.array_equal(mx1, mx2)
        # without duplicate edges random normal data has no ties: the winning
        # edge maps through p (with duplicates only the values must agree)
        keys = ei[0] * N + ei[1]
        if np.unique(keys).size == E:
            ok = a2 < E
            assert np.array_equal(p[a2[ok]], a1[ok]) and np.array_equal(a1[~ok], a2[~ok])
        iso = deg == 0
        for aggr in ("sum", "mean", "max"):
            o, a, _ = oracle.propagate(x, ei, w, aggr=aggr, lib=lib)
            assert (o[iso] == 0).all() and not np.signbit(o[iso]).any()
            if aggr == "max":
                assert (a[iso] == E).all()
        # diff mean = mean(x_j) - x_i where deg > 0
        md, _, _ = oracle.propagate(x, ei, msg="diff", aggr="mean", lib=lib)
        ms, _, _ = oracle.propagate(x, ei, aggr="mean", lib=lib)
        has = deg > 0
        assert np.allclose(md[has], ms[has] - x[has].astype(np.float64), rtol=1e-12, atol=1e-12)
    # block-diagonal batch = concatenation of per-graph results
    parts, xs, off = [], [], 0
    for n, e in ((5, 9), (1, 0), (8, 20), (3, 4)):
        parts.append(synth.random_coo(rng, n, e) + off)
        xs.append(rng.standard_normal((n, 3)).astype(np.float32))
        off += n
    ei = np.concatenate(parts, axis=1)
    x = np.concatenate(xs)
    for aggr in ("sum", "mean", "max"):
        whole, warg, _ = oracle.propagate(x, ei, aggr=aggr, lib=lib)
        off, eoff = 0, 0
        for pe, px in zip(parts, xs):
            n, e = px.shape[0], pe.shape[1]
            sub, sarg, _ = oracle.propagate(px, pe - off, aggr=aggr, lib=lib)
            assert np.array_equal(whole[off:off + n], sub)
            if aggr == "max":
                got = warg[off:off + n]
                assert np.array_equal(np.where(sarg == e, ei.shape[1], sarg + eoff), got)
            off += n
            eoff += e


def pin_pool_relations(lib):
    """Pooling equals propagate over the bipartite edges n -> N + batch[n];
    sum over graphs = column sums; one graph = a full reduction."""
    rng = np.random.default_rng(11)
    for sizes in ((3, 0, 4, 1), (1,), (10, 7, 0, 0, 2)):
        B = len(sizes)
        batch = np.repeat(np.arange(B), sizes).astype(np.int64)
        N = batch.size
        F = 3
        x = rng.standard_normal((N, F)).astype(np.float32)
        xe = np.concatenate([x, np.zeros((B, F), np.float32)])
        ei = np.stack([np.arange(N), N + batch]).astype(np.int64)
        for aggr in ("sum", "mean", "max"):
            out, arg, _ = oracle.global_pool(x, batch, B, aggr, lib=lib)
            ref, rarg, _ = oracle.propagate(xe, ei, aggr=aggr, lib=lib)
            assert np.array_equal(out, ref[N:])
            if aggr == "max":
                assert np.array_equal(arg, rarg[N:])
        s, _, _ = oracle.global_pool(x, batch, B, "sum", lib=lib)
        assert np.allclose(s.sum(axis=0), x.astype(np.float64).sum(axis=0), rtol=1e-12, atol=1e-12)
    x = rng.standard_normal((25, 4)).astype(np.float32)
    b = np.zeros(25, np.int64)
    out, _, _ = oracle.global_pool(x, b, 1, "mean", lib=lib)
    assert np.allclose(out[0], x.astype(np.float64).mean(axis=0), rtol=1e-12)
    out, arg, _ = oracle.global_pool(x, b, 1, "max", lib=lib)
    assert np.array_equal(out[0], x.max(axis=0)) and np.array_equal(arg[0], x.argmax(axis=0))


def pin_golden_backward(lib):
    g = golden()
    pr, b = g["propagate"], g["backward"]
    x = np.array(pr["x"], np.float32)
    ei = np.array(pr["edge_index"], np.int64)
    w = np.array(pr["edge_weight"], np.float32)
    go = np.array(b["grad_out"], np.float32)
    gx, _, _, _ = oracle.propagate_backward(x, ei, go, aggr="sum", lib=lib)
    assert np.array_equal(gx, np.array(b["sum_grad_x"]))
    gx, gw, _, _ = oracle.propagate_backward(x, ei, go, w, aggr="sum", want_grad_w=True, lib=lib)
    assert np.array_equal(gx, np.array(b["weighted_sum_grad_x"])) and np.array_equal(gw, np.array(b["weighted_sum_grad_w"]))
    gx, _, _, _ = oracle.propagate_backward(x, ei, go, aggr="mean", lib=lib)
    assert np.allclose(gx * 3.0, np.array(b["mean_grad_x_times_3"]), rtol=1e-15, atol=1e-15)
    gx, _, _, _ = oracle.propagate_backward(x, ei, go, aggr="max", argmax=np.array(pr["src_argmax"]), lib=lib)
    assert np.array_equal(gx, np.array(b["max_grad_x"]))
    gx, _, _, _ = oracle.propagate_backward(x, ei, go, msg="diff", aggr="sum", lib=lib)
    assert np.array_equal(gx, np.array(b["diff_sum_grad_x"]))


def _torch_forward(x, ei, w, msg, aggr, N):
    """An independent fp64 torch forward used only for its autograd."""
    src, dst = torch.from_numpy(ei[0]), torch.from_numpy(ei[1])
    if msg == "diff":
        m = x[src] - x[dst]
    else:
        m = x[src] * (w[:, None] if w is not None else 1.0)
    F = x.shape[1]
    if aggr == "max":
        base = torch.zeros(N, F, dtype=x.dtype)
        return base.scatter_reduce(0, dst[:, None].expand(-1, F), m, "amax", include_self=False)
    out = torch.zeros(N, F, dtype=x.dtype).index_add(0, dst, m)
    if aggr == "mean":
        deg = torch.bincount(dst, minlength=N).clamp(min=1).to(x.dtype)
        out = out / deg[:, None]
    return out


def pin_backward_autograd(lib):
    """torch autograd through an independent fp64 forward (tie-free data)."""
    rng = np.random.default_rng(31)
    for N, E in ((6, 14), (20, 90), (50, 300)):
        ei = synth.random_coo(rng, N, E, duplicates=False)
        F = 3
        x = rng.standard_normal((N, F)).astype(np.float32)
        w = rng.standard_normal(ei.shape[1]).astype(np.float32)
        go = rng.standard_normal((N, F)).astype(np.float32)
        for aggr in ("sum", "mean", "max"):
            for msg, weighted in (("src", False), ("src", True), ("diff", False)):
                xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
                wt = torch.tensor(w, dtype=torch.float64, requires_grad=True) if weighted else None
                out = _torch_forward(xt, ei, wt, msg, aggr, N)
                out.backward(torch.tensor(go, dtype=torch.float64))
                arg = None
                if aggr == "max":
                    _, arg, _ = oracle.propagate(x, ei, w if weighted else None, msg=msg, aggr="max", lib=lib)
                gx, gw, _, _ = oracle.propagate_backward(x, ei, go, w if weighted else None, msg=msg, aggr=aggr,
                                                         argmax=arg, want_grad_w=weighted, lib=lib)
                assert np.allclose(gx, xt.grad.numpy(), rtol=1e-9, atol=1e-9), (aggr, msg, weighted)
                if weighted:
                    assert np.allclose(gw, wt.grad.numpy(), rtol=1e-9, atol=1e-9), (aggr, msg)


def pin_backward_dense(lib):
    """Sum backward = A^T g (dense fp64 matmul); grad w_k = <g_i, x_j>."""
    for N, F, ei, x, w in small_cases():
        rng = np.random.default_rng(N)
        go = rng.standard_normal((N, F)).astype(np.float32)
        A = dense_adjacency(ei, N, w)
        gx, gw, sx, _ = oracle.propagate_backward(x, ei, go, w, aggr="sum", want_grad_w=True, lib=lib)
        assert np.allclose(gx, A.T @ go.astype(np.float64), rtol=1e-12, atol=1e-12)
        ref_w = (go.astype(np.float64)[ei[1]] * x.astype(np.float64)[ei[0]]).sum(axis=1)
        assert np.allclose(gw, ref_w, rtol=1e-12, atol=1e-12)


def _frac(a):
    a = np.asarray(a, np.float64)
    return a[..., 0] / a[..., 1]


def pin_golden_attention(lib):
    g = golden()["attention"]
    ei = np.array(g["edge_index"], np.int64)
    N, H = g["N"], g["H"]
    s = np.log(np.array(g["scores_log_of"], np.float64))
    s[:, 1] += g["head1_offset"]
    alpha = oracle.segment_softmax(s, ei, N, lib=lib)
    assert np.allclose(alpha, _frac(g["alpha_frac"]), rtol=1e-12, atol=0)
    e = oracle.gat_scores(np.array(g["a_src"]), np.array(g["a_dst"]), ei, g["slope"], lib=lib)
    assert np.array_equal(e, np.array(g["gat_scores"]))
    a32 = _frac(g["alpha_frac"]).astype(np.float32)
    gs, _ = oracle.segment_softmax_backward(a32, np.array(g["grad_alpha"]), ei, N, lib=lib)
    assert np.allclose(gs, _frac(g["softmax_grad_frac"]), rtol=1e-6, atol=1e-7)
    x = np.array(g["x"], np.float32)
    out, _ = oracle.propagate_heads(x, ei, a32, H, lib=lib)
    assert np.allclose(out, _frac(g["heads_out_frac"]), rtol=1e-6, atol=1e-7)
    gx, ga, _, _ = oracle.propagate_heads_backward(x, ei, a32, np.array(g["grad_out"]), H, lib=lib)
    assert np.allclose(gx, _frac(g["heads_grad_x_frac"]), rtol=1e-6, atol=1e-7)
    assert np.array_equal(ga, np.array(g["heads_grad_alpha"]))


def _attention_cases():
    """Random multigraphs with isolated targets and H in 1..4 heads."""
    rng = np.random.default_rng(4321)
    out = []
    for N, E, H in ((1, 3, 1), (5, 0, 2), (7, 20, 3), (16, 60, 1), (33, 200, 4), (64, 90, 2), (40, 300, 3)):
        ei = synth.random_coo(rng, N, E)
        s = (rng.standard_normal((E, H)) * 3.0).astype(np.float32)
        out.append((N, H, ei, s, rng))
    return out


def pin_softmax_library(lib):
    """Per-target softmax equals scipy.special.softmax of that target's scores."""
    from scipy.special import softmax
    for N, H, ei, s, _ in _attention_cases():
        alpha = oracle.segment_softmax(s, ei, N, lib=lib)
        for i in range(N):
            k = np.flatnonzero(ei[1] == i)
            if k.size:
                assert np.allclose(alpha[k], softmax(s[k].astype(np.float64), axis=0), rtol=1e-13, atol=1e-15)


def pin_softmax_invariants(lib):
    """Sums to one per (target, head); shift by a per-target constant changes
    nothing; one edge gives 1; two edges give the logistic function; edge
    order only permutes the result; no overflow at large scores."""
    from scipy.special import expit
    for N, H, ei, s, rng in _attention_cases():
        E = ei.shape[1]
        alpha = oracle.segment_softmax(s, ei, N, lib=lib)
        tot = np.zeros((N, H))
        np.add.at(tot, ei[1], alpha)
        has = np.bincount(ei[1], minlength=N) > 0
        assert np.allclose(tot[has], 1.0, rtol=0, atol=1e-13) and np.all(tot[~has] == 0)
        assert np.all(alpha > 0) and np.all(alpha <= 1)
        shift = rng.integers(-500, 500, size=(N, H)).astype(np.float64)
        shifted = oracle.segment_softmax(s.astype(np.float64) + shift[ei[1]], ei, N, lib=lib)
        assert np.allclose(shifted, alpha, rtol=1e-12, atol=1e-15)
        p = rng.permutation(E)
        assert np.allclose(oracle.segment_softmax(s[p], ei[:, p], N, lib=lib), alpha[p], rtol=1e-14, atol=0)
    ei = np.array([[0, 1, 2, 0], [1, 1, 2, 3]], np.int64)
    s = np.array([[2.5, 700.0], [-1.0, 699.0], [40.0, -40.0], [-3.0, 0.0]])
    alpha = oracle.segment_softmax(s, ei, 4, lib=lib)
    assert np.allclose(alpha[0], expit(s[0] - s[1]), rtol=1e-14, atol=0)
    assert np.allclose(alpha[1], expit(s[1] - s[0]), rtol=1e-14, atol=0)
    assert np.array_equal(alpha[2:], np.ones((2, 2)))


def _torch_softmax(s, dst, N):
    """An independent fp64 segment softmax in torch, used for its autograd."""
    H = s.shape[1]
    idx = dst[:, None].expand(-1, H)
    m = torch.full((N, H), -torch.inf, dtype=s.dtype).scatter_reduce(0, idx, s, "amax")
    ex = torch.exp(s - m[dst])
    den = torch.zeros(N, H, dtype=s.dtype).index_add(0, dst, ex)
    return ex / den[dst]


def pin_softmax_backward_autograd(lib):
    """torch autograd through an independent forward; gradients sum to zero
    over every segment (the softmax ignores a per-segment shift)."""
    for N, H, ei, s, rng in _attention_cases():
        E = ei.shape[1]
        dst = torch.from_numpy(ei[1])
        st = torch.tensor(s, dtype=torch.float64, requires_grad=True)
        alpha = _torch_softmax(st, dst, N)
        g = rng.standard_normal((E, H)).astype(np.float32)
        alpha.backward(torch.tensor(g, dtype=torch.float64))
        a32 = alpha.detach().numpy().astype(np.float32)
        gs, sabs = oracle.segment_softmax_backward(a32, g, ei, N, lib=lib)
        assert np.all(np.abs(gs - st.grad.numpy()) <= 1e-6 * sabs + 1e-12)
        tot = np.zeros((N, H))
        np.add.at(tot, ei[1], gs)
        tabs = np.zeros((N, H))
        np.add.at(tabs, ei[1], sabs)
        assert np.all(np.abs(tot) <= 1e-6 * tabs + 1e-12)


def pin_heads_dense(lib):
    """Per head, the attention sum is a dense matmul with the alpha-weighted
    adjacency; its backward is the transposed matmul and per-edge dots; one
    head equals the weighted propagate."""
    for N, H, ei, s, rng in _attention_cases():
        E = ei.shape[1]
        C = int(rng.integers(1, 4))
        x = rng.standard_normal((N, H * C)).astype(np.float32)
        a = rng.random((E, H)).astype(np.float32)
        g = rng.standard_normal((N, H * C)).astype(np.float32)
        out, _ = oracle.propagate_heads(x, ei, a, H, lib=lib)
        gx, ga, _, _ = oracle.propagate_heads_backward(x, ei, a, g, H, lib=lib)
        x64, g64 = x.astype(np.float64), g.astype(np.float64)
        for h in range(H):
            A = dense_adjacency(ei, N, a[:, h])
            cols = slice(h * C, (h + 1) * C)
            assert np.allclose(out[:, cols], A @ x64[:, cols], rtol=1e-12, atol=1e-12)
            assert np.allclose(gx[:, cols], A.T @ g64[:, cols], rtol=1e-12, atol=1e-12)
            ref = (g64[ei[1], cols] * x64[ei[0], cols]).sum(axis=1)
            assert np.allclose(ga[:, h], ref, rtol=1e-12, atol=1e-12)
        if H == 1:
            ref, _, _ = oracle.propagate(x, ei, a[:, 0], aggr="sum", lib=lib)
            assert np.array_equal(out, ref)


def pin_uniform_attention_is_mean(lib):
    """Equal scores give alpha = 1/deg, so the attention sum is the mean
    aggregation of every head's block."""
    for N, H, ei, _, rng in _attention_cases():
        E = ei.shape[1]
        a_node = np.zeros((N, H), np.float32)
        e = oracle.gat_scores(a_node, a_node, ei, 0.2, lib=lib)
        assert np.array_equal(e, np.zeros((E, H)))
        alpha = oracle.segment_softmax(e, ei, N, lib=lib)
        C = 2
        x = rng.standard_normal((N, H * C)).astype(np.float32)
        out, _ = oracle.propagate_heads(x, ei, alpha.astype(np.float32), H, lib=lib)
        mean, _, _ = oracle.propagate(x, ei, aggr="mean", lib=lib)
        assert np.allclose(out, mean, rtol=1e-6, atol=1e-6)


def pin_golden_dense_transform(lib):
    g = golden()["dense_transform"]
    out, sabs = oracle.dense_transform(np.array(g["x"]), np.array(g["theta"]), lib=lib)
    assert np.array_equal(out, np.array(g["out"]))
    assert np.array_equal(sabs, np.abs(np.array(g["x"])) @ np.abs(np.array(g["theta"])))


def pin_dense_transform_library(lib):
    """numpy matmul; identity and column-selector weights; and the GCN layer
    identity A (X Theta) = (A X) Theta across the propagate oracle."""
    rng = np.random.default_rng(71)
    for N, Fi, Fo in ((1, 1, 1), (5, 3, 7), (40, 16, 9), (33, 64, 32)):
        x = rng.standard_normal((N, Fi)).astype(np.float32)
        t = rng.standard_normal((Fi, Fo)).astype(np.float32)
        out, _ = oracle.dense_transform(x, t, lib=lib)
        assert np.allclose(out, x.astype(np.float64) @ t.astype(np.float64), rtol=1e-12, atol=1e-12)
        eye, _ = oracle.dense_transform(x, np.eye(Fi, dtype=np.float32), lib=lib)
        assert np.array_equal(eye, x.astype(np.float64))
    for N, F, ei, x, w in small_cases():
        t = np.random.default_rng(N).standard_normal((F, 4)).astype(np.float32)
        xt, _ = oracle.dense_transform(x, t, lib=lib)
        lhs, _, _ = oracle.propagate(xt.astype(np.float32), ei, w, aggr="sum", lib=lib)
        ax, _, _ = oracle.propagate(x, ei, w, aggr="sum", lib=lib)
        rhs = ax @ t.astype(np.float64)
        assert np.allclose(lhs, rhs, rtol=1e-5, atol=1e-5)


def pin_golden_edge_messages(lib):
    g = golden()
    pr, em = g["propagate"], g["edge_messages"]
    x = np.array(pr["x"], np.float32)
    ei = np.array(pr["edge_index"], np.int64)
    ea = np.array(em["edge_attr"], np.float32)
    for msg, key in (("edge_add", "add"), ("edge_relu", "relu"), ("edge_mul", "mul")):
        out, _, _ = oracle.propagate(x, ei, msg=msg, aggr="sum", edge_attr=ea, lib=lib)
        assert np.array_equal(out, np.array(em[f"{key}_sum"])), msg
        mean, _, _ = oracle.propagate(x, ei, msg=msg, aggr="mean", edge_attr=ea, lib=lib)
        assert np.allclose(mean * 3, np.array(em[f"{key}_sum"]), rtol=1e-15, atol=1e-15)
        mx, arg, _ = oracle.propagate(x, ei, msg=msg, aggr="max", edge_attr=ea, lib=lib)
        assert np.array_equal(mx, np.array(em[f"{key}_max"])) and np.array_equal(arg, np.array(em[f"{key}_argmax"])), msg


def pin_edge_messages_library(lib):
    """Sums against numpy scatter-adds of the formed messages, max against CPU
    torch scatter_reduce(amax); e = 0 (add) and e = 1 (mul) reduce to the plain
    propagate; large positive e makes relu the identity."""
    for N, F, ei, x, w in small_cases():
        rng = np.random.default_rng(N + 5)
        E = ei.shape[1]
        ea = rng.standard_normal((E, F)).astype(np.float32)
        xs = x[ei[0]].astype(np.float64)
        for msg, m in (("edge_add", xs + ea), ("edge_relu", np.maximum(xs + ea, 0.0)), ("edge_mul", xs * ea)):
            ref = np.zeros((N, F))
            np.add.at(ref, ei[1], m)
            out, _, _ = oracle.propagate(x, ei, msg=msg, aggr="sum", edge_attr=ea, lib=lib)
            assert np.allclose(out, ref, rtol=1e-12, atol=1e-12), msg
            mx, _, _ = oracle.propagate(x, ei, msg=msg, aggr="max", edge_attr=ea, lib=lib)
            m32 = torch.from_numpy(m.astype(np.float32))
            tmax = torch.zeros(N, F).scatter_reduce(0, torch.from_numpy(ei[1])[:, None].expand(-1, F), m32, "amax",
                                                    include_self=False)
            assert np.array_equal(mx.astype(np.float32), tmax.numpy()), msg
        for aggr in ("sum", "mean", "max"):
            base = oracle.propagate(x, ei, aggr=aggr, lib=lib)
            z = oracle.propagate(x, ei, msg="edge_add", aggr=aggr, edge_attr=np.zeros((E, F), np.float32), lib=lib)
            one = oracle.propagate(x, ei, msg="edge_mul", aggr=aggr, edge_attr=np.ones((E, F), np.float32), lib=lib)
            for got in (z, one):
                assert np.array_equal(got[0], base[0])
                if aggr == "max":
                    assert np.array_equal(got[1], base[1])
            big = np.full((E, F), 100.0, np.float32)
            r = oracle.propagate(x, ei, msg="edge_relu", aggr=aggr, edge_attr=big, lib=lib)
            a = oracle.propagate(x, ei, msg="edge_add", aggr=aggr, edge_attr=big, lib=lib)
            assert np.array_equal(r[0], a[0])


def pin_golden_gat_backward(lib):
    g = golden()["attention"]
    ei = np.array(g["edge_index"], np.int64)
    gs, gd, _, _ = oracle.gat_scores_backward(np.array(g["a_src"]), np.array(g["a_dst"]), ei,
                                              np.array(g["grad_scores"]), g["slope"], lib=lib)
    assert np.array_equal(gs, np.array(g["gat_grad_a_src"])) and np.array_equal(gd, np.array(g["gat_grad_a_dst"]))


def pin_gat_layer_autograd(lib):
    """A whole GAT attention layer (scores, softmax, attention sum) in CPU
    torch fp64 autograd against the oracle's backward chain: attention-sum
    backward -> softmax backward -> score backward."""
    for N, H, ei, _, rng in _attention_cases():
        E = ei.shape[1]
        C = 3
        x = rng.standard_normal((N, H * C)).astype(np.float32)
        a_src = rng.standard_normal((N, H)).astype(np.float32)
        a_dst = rng.standard_normal((N, H)).astype(np.float32)
        g = rng.standard_normal((N, H * C)).astype(np.float32)
        slope = 0.2
        src, dst = torch.from_numpy(ei[0]), torch.from_numpy(ei[1])
        xs = torch.tensor(x, dtype=torch.float64, requires_grad=True)
        at_s = torch.tensor(a_src, dtype=torch.float64, requires_grad=True)
        at_d = torch.tensor(a_dst, dtype=torch.float64, requires_grad=True)
        v = at_s[src] + at_d[dst]
        e = torch.where(v >= 0, v, slope * v)
        alpha = _torch_softmax(e, dst, N)
        msg = (alpha[:, :, None] * xs[src].view(E, H, C)).reshape(E, H * C)
        out = torch.zeros(N, H * C, dtype=torch.float64).index_add(0, dst, msg)
        out.backward(torch.tensor(g, dtype=torch.float64))
        # oracle chain in fp64 values rounded to fp32 where the kernels store fp32
        e_o = oracle.gat_scores(a_src, a_dst, ei, slope, lib=lib)
        al = oracle.segment_softmax(e_o, ei, N, lib=lib).astype(np.float32)
        gx, ga, _, sa = oracle.propagate_heads_backward(x, ei, al, g, H, lib=lib)
        gsc, ss = oracle.segment_softmax_backward(al, ga.astype(np.float32), ei, N, lib=lib)
        gs, gd, _, _ = oracle.gat_scores_backward(a_src, a_dst, ei, gsc.astype(np.float32), slope, lib=lib)
        assert np.allclose(gx, xs.grad.numpy(), rtol=1e-5, atol=1e-6)
        assert np.allclose(gs, at_s.grad.numpy(), rtol=1e-4, atol=1e-5)
        assert np.allclose(gd, at_d.grad.numpy(), rtol=1e-4, atol=1e-5)


def pin_golden_edge_backward(lib):
    g = golden()["edge_messages_backward"]
    ei = np.array(g["edge_index"], np.int64)
    x, ea, go = (np.array(g[k], np.float32) for k in ("x", "edge_attr", "grad_out"))
    for msg, key in (("edge_add", "add"), ("edge_relu", "relu"), ("edge_mul", "mul")):
        for aggr in ("sum", "mean", "max"):
            name = f"{key}_{aggr}"
            if name not in g:
                continue
            arg = None
            if aggr == "max":
                _, arg, _ = oracle.propagate(x, ei, msg=msg, aggr="max", edge_attr=ea, lib=lib)
                assert np.array_equal(arg, np.array(g[name]["argmax"])), name
            gx, ge, _, _ = oracle.propagate_edge_backward(x, ei, ea, go, msg, aggr, argmax=arg, lib=lib)
            assert np.array_equal(gx, np.array(g[name]["grad_x"], np.float64)), name
            assert np.array_equal(ge, np.array(g[name]["grad_e"], np.float64)), name


def pin_edge_backward_autograd(lib):
    """Every message and aggregation against CPU torch fp64 autograd of the
    forward written with index_add / scatter_reduce (max with distinct
    messages per row and column, so that autograd's split of tied maxima
    does not arise)."""
    for N, F, ei, x, _ in small_cases():
        E = ei.shape[1]
        rng = np.random.default_rng(N + 11)
        ea = rng.standard_normal((E, F)).astype(np.float32)
        g = rng.standard_normal((N, F)).astype(np.float32)
        src, dst = torch.from_numpy(ei[0]), torch.from_numpy(ei[1])
        deg = torch.bincount(dst, minlength=N).clamp(min=1).to(torch.float64)
        for msg in ("edge_add", "edge_relu", "edge_mul"):
            for aggr in ("sum", "mean", "max"):
                xs = torch.tensor(x, dtype=torch.float64, requires_grad=True)
                es = torch.tensor(ea, dtype=torch.float64, requires_grad=True)
                v = xs[src] + es if msg != "edge_mul" else xs[src] * es
                m = torch.relu(v) if msg == "edge_relu" else v
                if aggr == "max":
                    if msg == "edge_relu":  # zeros tie; keep the rows where every message is positive
                        continue
                    out = torch.zeros(N, F, dtype=torch.float64).scatter_reduce(
                        0, dst[:, None].expand(-1, F), m, "amax", include_self=False)
                else:
                    out = torch.zeros(N, F, dtype=torch.float64).index_add(0, dst, m)
                    if aggr == "mean":
                        out = out / deg[:, None]
                out.backward(torch.tensor(g, dtype=torch.float64))
                arg = None
                if aggr == "max":
                    _, arg, _ = oracle.propagate(x, ei, msg=msg, aggr="max", edge_attr=ea, lib=lib)
                gx, ge, _, _ = oracle.propagate_edge_backward(x, ei, ea, g, msg, aggr, argmax=arg, lib=lib)
                assert np.allclose(gx, xs.grad.numpy(), rtol=1e-12, atol=1e-12), (msg, aggr, N)
                assert np.allclose(ge, es.grad.numpy(), rtol=1e-12, atol=1e-12), (msg, aggr, N)


def pin_edge_backward_reductions(lib):
    """Special cases that reduce to the plain propagate backward: with e = 0
    the x-gradient of x_j + e, and with e = 1 that of x_j * e, is the plain
    sum/mean gradient; for x_j + e the feature gradient of every edge is
    its target's (scaled) upstream gradient; with e large and positive the
    relu gate is open everywhere."""
    for N, F, ei, x, _ in small_cases():
        E = ei.shape[1]
        g = np.random.default_rng(N + 13).standard_normal((N, F)).astype(np.float32)
        for aggr in ("sum", "mean"):
            base, _, _, _ = oracle.propagate_backward(x, ei, g, aggr=aggr, lib=lib)
            z = np.zeros((E, F), np.float32)
            # mean: g / deg here, g * (1 / deg) there: equal up to one rounding
            same = (lambda a, b: np.array_equal(a, b)) if aggr == "sum" else \
                (lambda a, b: np.allclose(a, b, rtol=0, atol=1e-12))
            gx, ge, _, _ = oracle.propagate_edge_backward(x, ei, z, g, "edge_add", aggr, lib=lib)
            assert same(gx, base), aggr
            deg = np.bincount(ei[1], minlength=N).astype(np.float64)
            dg = g.astype(np.float64)[ei[1]] / (np.maximum(deg, 1.0)[ei[1], None] if aggr == "mean" else 1.0)
            assert np.array_equal(ge, dg), aggr
            gx1, _, _, _ = oracle.propagate_edge_backward(x, ei, np.ones((E, F), np.float32), g, "edge_mul", aggr,
                                                         lib=lib)
            assert same(gx1, base), aggr
            big = np.full((E, F), 100.0, np.float32)
            r = oracle.propagate_edge_backward(x, ei, big, g, "edge_relu", aggr, lib=lib)
            a = oracle.propagate_edge_backward(x, ei, big, g, "edge_add", aggr, lib=lib)
            assert np.array_equal(r[0], a[0]) and np.array_equal(r[1], a[1]), aggr


ALL_PINS = [pin_golden_propagate, pin_golden_pool, pin_golden_gcn_norm, pin_golden_gcn_norm_directed,
            pin_golden_signed_zero,
            pin_degree_and_csr_library, pin_sum_mean_dense, pin_torch_scatter, pin_max_bruteforce,
            pin_gcn_norm_closed_forms, pin_invariants, pin_pool_relations, pin_golden_backward,
            pin_backward_autograd, pin_backward_dense, pin_golden_attention, pin_softmax_library,
            pin_softmax_invariants, pin_softmax_backward_autograd, pin_heads_dense, pin_uniform_attention_is_mean,
            pin_golden_dense_transform, pin_dense_transform_library, pin_golden_edge_messages,
            pin_edge_messages_library, pin_golden_gat_backward, pin_gat_layer_autograd, pin_golden_edge_backward,
            pin_edge_backward_autograd, pin_edge_backward_reductions]
