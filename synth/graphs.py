"""Seeded synthetic graph workloads shaped like the paper's benchmarks.

The paper's datasets are not available; these generators stand in for them
with the same shapes (Table 5 of the paper: Cora 2,708 nodes / 5,278 edges,
PubMed 19,717 / 44,324, small TU graphs of 10-40 nodes, ModelNet10 clouds of
1,024 points) plus one large power-law graph for bandwidth measurement.
No dataset item is reproduced; every value is drawn from a seeded numpy
generator.

Conventions: ``edge_index`` is int64 [2, E]; row 0 is the source, row 1 the
target of a directed edge. Undirected graphs are symmetrised into both
directions. Features are fp32 ~ N(0, 1), drawn after the graph from the same
generator.
"""
from __future__ import annotations

import numpy as np

CONFIG_NAMES = {
    1: "sparse-uniform N=2708 E=10556(+2708 self-loops) F=16",
    2: "power-law(Chung-Lu g=2.5) N=19717 E=88648+19717 F=64|500",
    3: "minibatch 128 ER graphs n~U[10,40] F=64",
    4: "knn clouds 16x1024 k=16 E=262144 F=64",
    5: "large power-law(Chung-Lu g=2.1) N=232965 E~114.6M+232965 F=128",
}


def rng_for(config: int, seed: int = 0) -> np.random.Generator:
    """Per-config generator: default_rng([seed, config])."""
    return np.random.default_rng([seed, config])


# ---------------------------------------------------------------- edge sets

def _dedupe_keep_first(keys: np.ndarray) -> np.ndarray:
    """Distinct values of ``keys`` in order of first occurrence."""
    _, first = np.unique(keys, return_index=True)
    return keys[np.sort(first)]


def uniform_pairs(N: int, M: int, rng: np.random.Generator) -> np.ndarray:
    """M distinct unordered pairs {u, v}, u != v, uniform over all pairs.
    Returns int64 [2, M] with u < v, in sampling order."""
    if M > N * (N - 1) // 2:
        raise ValueError("too many pairs")
    keys = np.empty(0, np.int64)
    while keys.size < M:
        need = M - keys.size
        n = int(need * 1.2) + 16
        u = rng.integers(0, N, n, dtype=np.int64)
        v = rng.integers(0, N, n, dtype=np.int64)
        ok = u != v
        lo, hi = np.minimum(u[ok], v[ok]), np.maximum(u[ok], v[ok])
        keys = _dedupe_keep_first(np.concatenate([keys, lo * N + hi]))
    keys = keys[:M]
    return np.stack([keys // N, keys % N])


def chung_lu_weights(N: int, gamma: float, total: float) -> np.ndarray:
    """Expected degrees w_i = c (i+1)^(-1/(gamma-1)), capped at sqrt(total)
    (the Chung-Lu condition that keeps pair probabilities <= 1), with c
    chosen by bisection so that sum(w) = total."""
    a = 1.0 / (gamma - 1.0)
    base = np.arange(1, N + 1, dtype=np.float64) ** (-a)
    cap = np.sqrt(total)
    lo, hi = 0.0, total
    for _ in range(200):
        c = 0.5 * (lo + hi)
        s = np.minimum(c * base, cap).sum()
        if s < total:
            lo = c
        else:
            hi = c
    return np.minimum(hi * base, cap)


def alias_table(p: np.ndarray):
    """Walker's alias table for sampling index i with probability p[i]."""
    n = p.size
    scaled = p * (n / p.sum())
    prob = np.ones(n)
    alias = np.arange(n, dtype=np.int64)
    small = list(np.nonzero(scaled < 1.0)[0])
    large = list(np.nonzero(scaled >= 1.0)[0])
    while small and large:
        s, l = small.pop(), large.pop()
        prob[s] = scaled[s]
        alias[s] = l
        scaled[l] -= 1.0 - scaled[s]
        (small if scaled[l] < 1.0 else large).append(l)
    return prob, alias


def alias_sample(prob: np.ndarray, alias: np.ndarray, n: int, rng: np.random.Generator) -> np.ndarray:
    idx = rng.integers(0, prob.size, n, dtype=np.int64)
    keep = rng.random(n) < prob[idx]
    return np.where(keep, idx, alias[idx])


def chung_lu_pairs(N: int, M: int, gamma: float, rng: np.random.Generator) -> np.ndarray:
    """M distinct unordered pairs sampled with endpoint probability
    proportional to the Chung-Lu expected degrees (self-pairs and repeats
    rejected, top-up rounds until M, a random subset dropped if over), then a
    random node relabelling so hubs are scattered over the id range.
    Returns int64 [2, M], u < v."""
    prob, alias = alias_table(chung_lu_weights(N, gamma, 2.0 * M))
    keys = np.empty(0, np.int64)
    while keys.size < M:
        need = M - keys.size
        n = int(need * 1.08) + 1024
        u = alias_sample(prob, alias, n, rng)
        v = alias_sample(prob, alias, n, rng)
        ok = u != v
        u, v = u[ok], v[ok]
        k = np.minimum(u, v) * N + np.maximum(u, v)
        del u, v, ok
        keys = np.unique(np.concatenate([keys, k]))
        del k
    if keys.size > M:
        drop = rng.choice(keys.size, keys.size - M, replace=False)
        mask = np.ones(keys.size, bool)
        mask[drop] = False
        keys = keys[mask]
    relabel = rng.permutation(N).astype(np.int64)
    lo, hi = np.divmod(keys, N)
    del keys
    out = np.empty((2, M), np.int64)
    np.take(relabel, lo, out=out[0])
    np.take(relabel, hi, out=out[1])
    return out


def symmetrize(pairs: np.ndarray) -> np.ndarray:
    """Both directions of every undirected pair: [u->v ..., v->u ...]."""
    M = pairs.shape[1]
    out = np.empty((2, 2 * M), np.int64)
    out[0, :M], out[0, M:] = pairs[0], pairs[1]
    out[1, :M], out[1, M:] = pairs[1], pairs[0]
    return out


def with_self_loops(edge_index: np.ndarray, N: int) -> np.ndarray:
    """Append the N self-loops (i, i) after the existing edges."""
    E = edge_index.shape[1]
    out = np.empty((2, E + N), np.int64)
    out[:, :E] = edge_index
    out[0, E:] = np.arange(N, dtype=np.int64)
    out[1, E:] = out[0, E:]
    return out


def shuffle_edges(edge_index: np.ndarray, rng: np.random.Generator) -> np.ndarray:
    """Random edge order (one uniform permutation applied to both rows)."""
    p = rng.permutation(edge_index.shape[1])
    out = np.empty((2, p.size), np.int64)
    np.take(edge_index[0], p, out=out[0])
    np.take(edge_index[1], p, out=out[1])
    return out


def features(N: int, F: int, rng: np.random.Generator) -> np.ndarray:
    return rng.standard_normal((N, F), dtype=np.float32)


# ------------------------------------------------------- small test graphs

def random_coo(rng: np.random.Generator, N: int, E: int, self_loops: bool = True,
               duplicates: bool = True) -> np.ndarray:
    """Arbitrary directed multigraph: E edges with uniform endpoints."""
    src = rng.integers(0, N, E, dtype=np.int64)
    dst = rng.integers(0, N, E, dtype=np.int64)
    if not self_loops:
        bad = src == dst
        while bad.any():
            src[bad] = rng.integers(0, N, int(bad.sum()), dtype=np.int64)
            bad = src == dst
    ei = np.stack([src, dst])
    if not duplicates and E:
        k = _dedupe_keep_first(src * N + dst)
        ei = np.stack([k // N, k % N])
    return np.ascontiguousarray(ei)


def graded_in_degree(rng: np.random.Generator, N: int, degrees) -> np.ndarray:
    """Targets 0 .. len(degrees)-1 receive degrees[i] edges each from
    uniform random sources in [0, N); edges in random order. Row lengths
    spread over a chosen range (short rows, rows of a few hundred to a few
    thousand slots, ...) without one hub taking the graph."""
    deg = np.asarray(degrees, dtype=np.int64)
    dst = np.repeat(np.arange(deg.size, dtype=np.int64), deg)
    src = rng.integers(0, N, dst.size, dtype=np.int64)
    order = rng.permutation(dst.size)
    return np.ascontiguousarray(np.stack([src[order], dst[order]]))


def star_graph(N: int, hub: int = 0, rng: np.random.Generator | None = None) -> np.ndarray:
    """Every other node points at ``hub`` (one in-degree N-1 row)."""
    leaves = np.array([i for i in range(N) if i != hub], np.int64)
    ei = np.stack([leaves, np.full_like(leaves, hub)])
    return shuffle_edges(ei, rng) if rng is not None else ei


def erdos_renyi(N: int, avg_degree: float, rng: np.random.Generator, coalesced: bool = False) -> np.ndarray:
    """Directed Erdos-Renyi G(n, m) graph: m = round(N * avg_degree) distinct
    pairs j -> i, j != i, uniform over all such pairs. `coalesced` orders the
    edges by target (the CSR row), ascending source inside a target;
    otherwise the order is random."""
    M = int(round(N * avg_degree))
    if M > N * (N - 1):
        raise ValueError("too many edges")
    keys = np.empty(0, np.int64)
    while keys.size < M:
        n = int((M - keys.size) * 1.1) + 16
        j = rng.integers(0, N, n, dtype=np.int64)
        i = rng.integers(0, N, n, dtype=np.int64)
        ok = j != i
        keys = _dedupe_keep_first(np.concatenate([keys, i[ok] * N + j[ok]]))
    keys = keys[:M]
    if coalesced:
        keys = np.sort(keys)
    else:
        keys = keys[rng.permutation(M)]
    return np.ascontiguousarray(np.stack([keys % N, keys // N]))


# ----------------------------------------------------------------- configs

def config1_sparse_uniform(seed: int = 0):
    """Cora-shaped sparse uniform graph: 2,708 nodes, 5,278 undirected pairs."""
    rng = rng_for(1, seed)
    N, F = 2708, 16
    ei = shuffle_edges(symmetrize(uniform_pairs(N, 5278, rng)), rng)
    x = features(N, F, rng)
    return {"name": CONFIG_NAMES[1], "N": N, "F": F, "edge_index": ei,
            "edge_index_gcn": with_self_loops(ei, N), "x": x}


def config2_power_law(seed: int = 0, F: int = 64):
    """PubMed-shaped power-law graph: Chung-Lu gamma=2.5, 19,717 nodes,
    44,324 undirected pairs, plus self-loops, in random edge order."""
    rng = rng_for(2, seed)
    N = 19717
    ei = symmetrize(chung_lu_pairs(N, 44324, 2.5, rng))
    ei_gcn = shuffle_edges(with_self_loops(ei, N), rng)
    x64 = features(N, 64, rng)
    x500 = features(N, 500, rng)
    return {"name": CONFIG_NAMES[2], "N": N, "F": F, "edge_index": shuffle_edges(ei, rng),
            "edge_index_gcn": ei_gcn, "x": x64 if F == 64 else x500, "x64": x64, "x500": x500}


def config3_minibatch(seed: int = 0):
    """128 small Erdos-Renyi graphs, n ~ U[10, 40], 2.2 undirected edges per
    node on average, packed block-diagonally with a batch vector."""
    rng = rng_for(3, seed)
    G, F = 128, 64
    sizes = rng.integers(10, 41, G)
    parts, offset = [], 0
    for n in sizes:
        n = int(n)
        p = min(1.0, 4.4 / (n - 1))
        iu, ju = np.triu_indices(n, 1)
        keep = rng.random(iu.size) < p
        pairs = np.stack([iu[keep], ju[keep]]).astype(np.int64)
        parts.append(symmetrize(pairs) + offset)
        offset += n
    N = offset
    ei = np.ascontiguousarray(np.concatenate(parts, axis=1))
    batch = np.repeat(np.arange(G, dtype=np.int64), sizes)
    x = features(N, F, rng)
    return {"name": CONFIG_NAMES[3], "N": N, "F": F, "B": G, "edge_index": ei, "batch": batch,
            "sizes": sizes.astype(np.int64), "x": x}


def config4_knn_clouds(seed: int = 0):
    """16 clouds x 1,024 points uniform in the unit ball; per-cloud directed
    k=16 nearest-neighbour graph (squared Euclidean in fp64, self excluded,
    ties to the lower index), edges neighbour -> centre."""
    rng = rng_for(4, seed)
    C, P, K, F = 16, 1024, 16, 64
    srcs, dsts = [], []
    for c in range(C):
        d = rng.standard_normal((P, 3))
        d /= np.linalg.norm(d, axis=1, keepdims=True)
        pts = d * rng.random((P, 1)) ** (1.0 / 3.0)
        sq = ((pts[:, None, :] - pts[None, :, :]) ** 2).sum(-1)
        np.fill_diagonal(sq, np.inf)
        nbr = np.argsort(sq, axis=1, kind="stable")[:, :K]
        srcs.append(nbr.reshape(-1) + c * P)
        dsts.append(np.repeat(np.arange(P), K) + c * P)
    ei = np.stack([np.concatenate(srcs), np.concatenate(dsts)]).astype(np.int64)
    x = features(C * P, F, rng)
    return {"name": CONFIG_NAMES[4], "N": C * P, "F": F, "edge_index": np.ascontiguousarray(ei),
            "edge_index_shuffled": shuffle_edges(ei, rng), "x": x}


def config5_large_power_law(seed: int = 0, pairs: int = 57_300_000, N: int = 232965, F: int = 128):
    """Large power-law graph: Chung-Lu gamma=2.1, mean degree ~492,
    114.6M directed edges plus N self-loops, random edge order."""
    rng = rng_for(5, seed)
    ei = with_self_loops(symmetrize(chung_lu_pairs(N, pairs, 2.1, rng)), N)
    ei = shuffle_edges(ei, rng)
    x = features(N, F, rng)
    return {"name": CONFIG_NAMES[5], "N": N, "F": F, "edge_index_gcn": ei, "x": x}


def make_config(i: int, seed: int = 0, **kw):
    return {1: config1_sparse_uniform, 2: config2_power_law, 3: config3_minibatch,
            4: config4_knn_clouds, 5: config5_large_power_law}[i](seed, **kw)
