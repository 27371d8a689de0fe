"""Oracle: plain CPU definition of the propagate path (test infrastructure).

This package is TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it. The HIP library
and its Python binding never import it, and it imports nothing from them.

The arithmetic lives in ``oracle.c`` (plain C loops, fp64 accumulation),
compiled with gcc into ``liboracle.so``. This module only marshals numpy
arrays through ctypes. Every function follows Eq. (1) of the paper
(Section 2, "Neighborhood Aggregation") with gamma = identity, or the
"Global Pooling" / "Mini-batch Handling" paragraphs of Section 2, or the
attention operator GAT named there, whose sparse softmax Section 3 (runtime
paragraph) singles out.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

MSG = {"src": 0, "diff": 1, "edge_add": 2, "edge_relu": 3, "edge_mul": 4}
AGGR = {"sum": 0, "mean": 1, "max": 2}
_ERR = {-1: "invalid argument", -2: "index out of range", -3: "non-finite input"}

_lib = None


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-fPIC",
           "-shared", "-Wall", "-Werror", src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def load(path: str | None = None) -> ctypes.CDLL:
    """Load a compiled oracle library; build the default one if absent."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        _lib = _bind(ctypes.CDLL(_LIB_PATH))
    return _lib


def _bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    p, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.oracle_degree.argtypes = [p, i64, i64, p]
    lib.oracle_coo_to_csr.argtypes = [p, i64, i64, p, p, p]
    lib.oracle_gcn_norm.argtypes = [p, p, i64, i64, p]
    lib.oracle_propagate.argtypes = [p, i64, i64, p, i64, p, p, i32, i32, p, p, p]
    lib.oracle_global_pool.argtypes = [p, i64, i64, p, i64, i32, p, p, p]
    lib.oracle_propagate_backward.argtypes = [p, i64, i64, p, i64, p, i32, i32, p, p, p, p, p, p]
    lib.oracle_propagate_edge_backward.argtypes = [p, i64, i64, p, i64, p, i32, i32, p, p, p, p, p, p]
    lib.oracle_gat_scores.argtypes = [p, p, i64, i64, p, i64, ctypes.c_float, p]
    lib.oracle_segment_softmax.argtypes = [p, i64, i64, p, i64, p]
    lib.oracle_segment_softmax_backward.argtypes = [p, p, i64, i64, p, i64, p, p]
    lib.oracle_propagate_heads.argtypes = [p, i64, i64, i64, p, i64, p, p, p]
    lib.oracle_propagate_heads_backward.argtypes = [p, i64, i64, i64, p, i64, p, p, p, p, p, p]
    lib.oracle_dense_transform.argtypes = [p, i64, i64, p, i64, p, p]
    lib.oracle_gat_scores_backward.argtypes = [p, p, i64, i64, p, i64, ctypes.c_float, p, p, p, p, p]
    for fn in (lib.oracle_degree, lib.oracle_coo_to_csr, lib.oracle_gcn_norm,
               lib.oracle_propagate, lib.oracle_global_pool, lib.oracle_propagate_backward,
               lib.oracle_gat_scores, lib.oracle_segment_softmax, lib.oracle_segment_softmax_backward,
               lib.oracle_propagate_heads, lib.oracle_propagate_heads_backward, lib.oracle_dense_transform,
               lib.oracle_gat_scores_backward):
        fn.restype = ctypes.c_int
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what}: {_ERR.get(rc, rc)}")


def _ei(edge_index) -> np.ndarray:
    ei = np.ascontiguousarray(edge_index, dtype=np.int64)
    if ei.ndim != 2 or ei.shape[0] != 2:
        raise ValueError("edge_index must be [2, E]")
    return ei


def degree(edge_index, N: int, lib=None) -> np.ndarray:
    """In-degree of every node: incoming edges counted with multiplicity."""
    lib = lib or load()
    ei = _ei(edge_index)
    deg = np.empty(N, np.int64)
    _check(lib.oracle_degree(_ptr(ei), ei.shape[1], N, _ptr(deg)), "degree")
    return deg


def coo_to_csr(edge_index, N: int, lib=None):
    """Stable target-sorted CSR: (rowptr [N+1], col [E], perm [E]), all int64."""
    lib = lib or load()
    ei = _ei(edge_index)
    E = ei.shape[1]
    rowptr = np.empty(N + 1, np.int64)
    col = np.empty(E, np.int64)
    perm = np.empty(E, np.int64)
    _check(lib.oracle_coo_to_csr(_ptr(ei), E, N, _ptr(rowptr), _ptr(col), _ptr(perm)), "coo_to_csr")
    return rowptr, col, perm


def gcn_norm(edge_index, N: int, edge_weight=None, lib=None) -> np.ndarray:
    """fp64 GCN edge normalisation dinv_j * w_k * dinv_i (self-loops already present)."""
    lib = lib or load()
    ei = _ei(edge_index)
    E = ei.shape[1]
    w = None if edge_weight is None else np.ascontiguousarray(edge_weight, dtype=np.float64)
    norm = np.empty(E, np.float64)
    _check(lib.oracle_gcn_norm(_ptr(ei), _ptr(w), E, N, _ptr(norm)), "gcn_norm")
    return norm


def propagate(x, edge_index, edge_weight=None, msg: str = "src", aggr: str = "sum", lib=None, edge_attr=None):
    """Eq. (1) with gamma = identity. Returns (out fp64 [N,F], argmax int64 [N,F] or None,
    sabs fp64 [N,F] = sum |message| (per degree for mean)). edge_attr [E, F]
    goes with the edge_* messages."""
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim != 2:
        raise ValueError("x must be [N, F]")
    N, F = x.shape
    ei = _ei(edge_index)
    E = ei.shape[1]
    w = None if edge_weight is None else np.ascontiguousarray(edge_weight, dtype=np.float32)
    ea = None if edge_attr is None else np.ascontiguousarray(edge_attr, dtype=np.float32)
    if ea is not None and ea.shape != (E, F):
        raise ValueError("edge_attr must be [E, F]")
    out = np.empty((N, F), np.float64)
    sabs = np.empty((N, F), np.float64)
    arg = np.empty((N, F), np.int64) if aggr == "max" else None
    _check(lib.oracle_propagate(_ptr(x), N, F, _ptr(ei), E, _ptr(w), _ptr(ea), MSG[msg], AGGR[aggr],
                                _ptr(out), _ptr(arg), _ptr(sabs)), "propagate")
    return out, arg, sabs


def global_pool(x, batch, B: int, aggr: str = "sum", lib=None):
    """Per-graph readout over a non-decreasing assignment vector.
    Returns (out fp64 [B,F], argmax node id int64 [B,F] or None, sabs)."""
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    N, F = x.shape
    batch = np.ascontiguousarray(batch, dtype=np.int64)
    if batch.shape != (N,):
        raise ValueError("batch must be [N]")
    out = np.empty((B, F), np.float64)
    sabs = np.empty((B, F), np.float64)
    arg = np.empty((B, F), np.int64) if aggr == "max" else None
    _check(lib.oracle_global_pool(_ptr(x), N, F, _ptr(batch), B, AGGR[aggr], _ptr(out),
                                  _ptr(arg), _ptr(sabs)), "global_pool")
    return out, arg, sabs


def propagate_backward(x, edge_index, grad_out, edge_weight=None, msg: str = "src", aggr: str = "sum",
                       argmax=None, want_grad_w: bool = False, lib=None):
    """Gradient of propagate for the upstream gradient grad_out. argmax is the
    forward's (max only). Returns (grad_x fp64 [N,F], grad_w fp64 [E] or None,
    sabs_x, sabs_w)."""
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    N, F = x.shape
    g = np.ascontiguousarray(grad_out, dtype=np.float32)
    if g.shape != (N, F):
        raise ValueError("grad_out must be [N, F]")
    ei = _ei(edge_index)
    E = ei.shape[1]
    w = None if edge_weight is None else np.ascontiguousarray(edge_weight, dtype=np.float32)
    arg = None if argmax is None else np.ascontiguousarray(argmax, dtype=np.int64)
    gx = np.empty((N, F), np.float64)
    sx = np.empty((N, F), np.float64)
    gw = np.empty(E, np.float64) if want_grad_w else None
    sw = np.empty(E, np.float64) if want_grad_w else None
    _check(lib.oracle_propagate_backward(_ptr(x), N, F, _ptr(ei), E, _ptr(w), MSG[msg], AGGR[aggr], _ptr(g),
                                         _ptr(arg), _ptr(gx), _ptr(gw), _ptr(sx), _ptr(sw)), "propagate_backward")
    return gx, gw, sx, sw


def propagate_edge_backward(x, edge_index, edge_attr, grad_out, msg: str, aggr: str = "sum", argmax=None,
                            want_grad_x: bool = True, want_grad_e: bool = True, lib=None):
    """Gradient of propagate with an edge-feature message ("edge_add",
    "edge_relu", "edge_mul") with respect to x and to the edge features
    (COO edge order). argmax is the forward's (max only). Returns (grad_x fp64
    [N,F] or None, grad_e fp64 [E,F] or None, sabs_x, sabs_e)."""
    lib = lib or load()
    if msg not in ("edge_add", "edge_relu", "edge_mul"):
        raise ValueError("msg must be an edge-feature message")
    x = np.ascontiguousarray(x, dtype=np.float32)
    N, F = x.shape
    g = np.ascontiguousarray(grad_out, dtype=np.float32)
    if g.shape != (N, F):
        raise ValueError("grad_out must be [N, F]")
    ei = _ei(edge_index)
    E = ei.shape[1]
    ea = np.ascontiguousarray(edge_attr, dtype=np.float32)
    if ea.shape != (E, F):
        raise ValueError("edge_attr must be [E, F]")
    arg = None if argmax is None else np.ascontiguousarray(argmax, dtype=np.int64)
    gx = np.empty((N, F), np.float64) if want_grad_x else None
    sx = np.empty((N, F), np.float64) if want_grad_x else None
    ge = np.empty((E, F), np.float64) if want_grad_e else None
    se = np.empty((E, F), np.float64) if want_grad_e else None
    _check(lib.oracle_propagate_edge_backward(_ptr(x), N, F, _ptr(ei), E, _ptr(ea), MSG[msg], AGGR[aggr], _ptr(g),
                                              _ptr(arg), _ptr(gx), _ptr(ge), _ptr(sx), _ptr(se)),
           "propagate_edge_backward")
    return gx, ge, sx, se


def _scores2d(a, E: int, name: str, dtype=np.float32) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=dtype)
    if a.ndim == 1:
        a = a.reshape(E, 1)
    if a.ndim != 2 or a.shape[0] != E:
        raise ValueError(f"{name} must be [E, H]")
    return a


def gat_scores(a_src, a_dst, edge_index, slope: float = 0.2, lib=None) -> np.ndarray:
    """GAT edge scores LeakyReLU(a_src[j] + a_dst[i]) per head, fp64 [E, H]."""
    lib = lib or load()
    a_src = np.ascontiguousarray(a_src, dtype=np.float32)
    a_dst = np.ascontiguousarray(a_dst, dtype=np.float32)
    if a_src.ndim != 2 or a_src.shape != a_dst.shape:
        raise ValueError("a_src and a_dst must both be [N, H]")
    N, H = a_src.shape
    ei = _ei(edge_index)
    E = ei.shape[1]
    e = np.empty((E, H), np.float64)
    _check(lib.oracle_gat_scores(_ptr(a_src), _ptr(a_dst), N, H, _ptr(ei), E, ctypes.c_float(slope), _ptr(e)),
           "gat_scores")
    return e


def segment_softmax(scores, edge_index, N: int, lib=None) -> np.ndarray:
    """Softmax of the scores [E, H] (or [E]) over the incoming edges of each
    target, per head; fp64 [E, H]."""
    lib = lib or load()
    ei = _ei(edge_index)
    E = ei.shape[1]
    s = _scores2d(scores, E, "scores", np.float64)
    H = s.shape[1]
    alpha = np.empty((E, H), np.float64)
    _check(lib.oracle_segment_softmax(_ptr(s), E, H, _ptr(ei), N, _ptr(alpha)), "segment_softmax")
    return alpha


def segment_softmax_backward(alpha, grad, edge_index, N: int, lib=None):
    """Gradient of segment_softmax w.r.t. its scores. Returns (grad_s fp64 [E, H], sabs)."""
    lib = lib or load()
    ei = _ei(edge_index)
    E = ei.shape[1]
    a = _scores2d(alpha, E, "alpha")
    g = _scores2d(grad, E, "grad")
    if g.shape != a.shape:
        raise ValueError("grad must match alpha")
    H = a.shape[1]
    gs = np.empty((E, H), np.float64)
    sabs = np.empty((E, H), np.float64)
    _check(lib.oracle_segment_softmax_backward(_ptr(a), _ptr(g), E, H, _ptr(ei), N, _ptr(gs), _ptr(sabs)),
           "segment_softmax_backward")
    return gs, sabs


def propagate_heads(x, edge_index, alpha, H: int, lib=None):
    """Sum over incoming edges of alpha[k, h] * x_j[h-th block of C columns];
    x is [N, H*C]. Returns (out fp64 [N, H*C], sabs)."""
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    N, F = x.shape
    if H <= 0 or F % H:
        raise ValueError("the feature width must be a multiple of H")
    ei = _ei(edge_index)
    E = ei.shape[1]
    a = _scores2d(alpha, E, "alpha")
    if a.shape[1] != H:
        raise ValueError("alpha must be [E, H]")
    out = np.empty((N, F), np.float64)
    sabs = np.empty((N, F), np.float64)
    _check(lib.oracle_propagate_heads(_ptr(x), N, H, F // H, _ptr(ei), E, _ptr(a), _ptr(out), _ptr(sabs)),
           "propagate_heads")
    return out, sabs


def propagate_heads_backward(x, edge_index, alpha, grad_out, H: int, lib=None):
    """Gradient of propagate_heads. Returns (grad_x fp64 [N, H*C], grad_alpha fp64 [E, H],
    sabs_x, sabs_alpha)."""
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    N, F = x.shape
    if H <= 0 or F % H:
        raise ValueError("the feature width must be a multiple of H")
    g = np.ascontiguousarray(grad_out, dtype=np.float32)
    if g.shape != (N, F):
        raise ValueError("grad_out must be [N, F]")
    ei = _ei(edge_index)
    E = ei.shape[1]
    a = _scores2d(alpha, E, "alpha")
    if a.shape[1] != H:
        raise ValueError("alpha must be [E, H]")
    gx = np.empty((N, F), np.float64)
    sx = np.empty((N, F), np.float64)
    ga = np.empty((E, H), np.float64)
    sa = np.empty((E, H), np.float64)
    _check(lib.oracle_propagate_heads_backward(_ptr(x), N, H, F // H, _ptr(ei), E, _ptr(a), _ptr(g), _ptr(gx),
                                               _ptr(ga), _ptr(sx), _ptr(sa)), "propagate_heads_backward")
    return gx, ga, sx, sa


def dense_transform(x, theta, lib=None):
    """X Theta of a GCN layer in fp64. Returns (out [N, Fo], sabs)."""
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    t = np.ascontiguousarray(theta, dtype=np.float32)
    if x.ndim != 2 or t.ndim != 2 or x.shape[1] != t.shape[0]:
        raise ValueError("x must be [N, Fi] and theta [Fi, Fo]")
    N, Fi = x.shape
    Fo = t.shape[1]
    out = np.empty((N, Fo), np.float64)
    sabs = np.empty((N, Fo), np.float64)
    _check(lib.oracle_dense_transform(_ptr(x), N, Fi, _ptr(t), Fo, _ptr(out), _ptr(sabs)), "dense_transform")
    return out, sabs


def gat_scores_backward(a_src, a_dst, edge_index, grad_e, slope: float = 0.2, lib=None):
    """Gradient of gat_scores for dL/d e [E, H]. Returns (grad_a_src fp64 [N, H],
    grad_a_dst fp64 [N, H], sabs_src, sabs_dst)."""
    lib = lib or load()
    a_src = np.ascontiguousarray(a_src, dtype=np.float32)
    a_dst = np.ascontiguousarray(a_dst, dtype=np.float32)
    if a_src.ndim != 2 or a_src.shape != a_dst.shape:
        raise ValueError("a_src and a_dst must both be [N, H]")
    N, H = a_src.shape
    ei = _ei(edge_index)
    E = ei.shape[1]
    g = _scores2d(grad_e, E, "grad_e")
    if g.shape[1] != H:
        raise ValueError("grad_e must be [E, H]")
    gs, gd = np.empty((N, H)), np.empty((N, H))
    ss, sd = np.empty((N, H)), np.empty((N, H))
    _check(lib.oracle_gat_scores_backward(_ptr(a_src), _ptr(a_dst), N, H, _ptr(ei), E, ctypes.c_float(slope), _ptr(g),
                                          _ptr(gs), _ptr(gd), _ptr(ss), _ptr(sd)), "gat_scores_backward")
    return gs, gd, ss, sd
