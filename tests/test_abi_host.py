"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any device work."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pyg_mi355x.h")

PYG_OK, INVALID, WORKSPACE, UNSUPPORTED = 0, -1, -3, -5
FAKE = ctypes.c_void_p(0x10000)  # never dereferenced: every call below fails its host checks


@pytest.fixture(scope="module")
def lib():
    import paper_1903_02428_amd as pyg
    if not os.path.exists(pyg.library_path()):
        from paper_1903_02428_amd import build
        build.build()
    return pyg.library()


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(pyg_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), f"{n} declared in the header but not exported"
    import paper_1903_02428_amd.binding as b
    assert sorted(b.EXPORTED) == names


def test_version_and_strerror(lib):
    import paper_1903_02428_amd as pyg
    assert pyg.abi_version() == 2
    for code, text in ((0, "success"), (-1, "invalid argument"), (-3, "workspace too small"),
                       (-4, "HIP runtime or launch error"), (-5, "unsupported size or combination"), (7, "unknown status")):
        assert pyg.strerror(code) == text


def _ws(fn, *args):
    out = ctypes.c_size_t(0)
    rc = fn(*args, ctypes.byref(out))
    return rc, out.value


def test_workspace_queries_monotone(lib):
    last = 0
    for E in (0, 1, 1000, 10**6, 10**8):
        rc, b = _ws(lib.pyg_coo_to_csr_workspace, E, 5000)
        assert rc == PYG_OK and b >= last
        last = b
    last = 0
    for N in (1, 100, 10**5):
        rc, b = _ws(lib.pyg_gcn_norm_workspace, 1000, N)
        assert rc == PYG_OK and b >= N * 8 and b >= last
        last = b
    for kernel in (0, 1, 2):
        for aggr in (0, 1, 2):
            last = 0
            for E in (0, 100, 10**5, 10**7):
                rc, b = _ws(lib.pyg_propagate_workspace, 0, 1000, 64, E, aggr, kernel, 0)
                assert rc == PYG_OK and b >= last
                last = b
    assert _ws(lib.pyg_propagate_workspace, 5, 10, 4, 10, 0, 0, 0)[0] == INVALID  # bad dtype
    assert _ws(lib.pyg_propagate_workspace, 0, 10, 4, 10, 9, 0, 0)[0] == INVALID  # bad aggr
    assert _ws(lib.pyg_propagate_workspace, 0, 2**31, 4, 10, 0, 0, 0)[0] == UNSUPPORTED
    assert _ws(lib.pyg_coo_to_csr_workspace, -1, 4)[0] == INVALID


def prop(lib, x=FAKE, dtype=0, N=10, F=4, ei=FAKE, E=20, w=None, csr=None, msg=0, aggr=0, kernel=1,
         out=ctypes.c_void_p(0x20000), argmax=None, ws=FAKE, ws_bytes=1 << 40):
    return lib.pyg_propagate(x, dtype, N, F, ei, E, w, csr, msg, aggr, kernel, out, argmax, ws, ws_bytes, None)


def test_propagate_rejects_bad_arguments(lib):
    from paper_1903_02428_amd.binding import _Csr
    assert prop(lib, dtype=3) == INVALID
    assert prop(lib, aggr=7) == INVALID
    assert prop(lib, msg=4) == INVALID
    assert prop(lib, kernel=9) == INVALID
    assert prop(lib, N=-1) == INVALID
    assert prop(lib, F=-2) == INVALID
    assert prop(lib, E=-5) == INVALID
    assert prop(lib, N=2**31) == UNSUPPORTED
    assert prop(lib, E=2**31) == UNSUPPORTED
    assert prop(lib, msg=1, w=FAKE) == INVALID                        # weighted diff
    assert prop(lib, aggr=2, argmax=None) == INVALID                  # max needs argmax
    assert prop(lib, aggr=0, argmax=ctypes.c_void_p(0x90000)) == INVALID  # argmax only for max
    assert prop(lib, x=None) == INVALID
    assert prop(lib, out=None) == INVALID
    assert prop(lib, ei=None) == INVALID                              # COO kernel needs edges
    assert prop(lib, N=0, E=5) == INVALID                             # edges into no nodes
    assert prop(lib, out=ctypes.c_void_p(0x10000 + 8)) == INVALID     # out overlaps x
    assert prop(lib, kernel=2, csr=None) == INVALID                   # CSR kernel needs a CSR
    bad_n = _Csr(0x30000, 0x40000, 0x50000, None, 11, 20, 0)
    assert prop(lib, kernel=2, csr=ctypes.byref(bad_n)) == INVALID    # CSR of another graph
    no_w = _Csr(0x30000, 0x40000, 0x50000, None, 10, 20, 0)
    assert prop(lib, kernel=2, csr=ctypes.byref(no_w), w=FAKE) == INVALID  # weights missing in CSR
    no_perm = _Csr(0x30000, 0x40000, None, None, 10, 20, 0)
    assert prop(lib, kernel=2, csr=ctypes.byref(no_perm), aggr=2, argmax=ctypes.c_void_p(0x90000)) == INVALID
    neg_chunk = _Csr(0x30000, 0x40000, 0x50000, None, 10, 20, -1)
    assert prop(lib, kernel=2, csr=ctypes.byref(neg_chunk)) == INVALID
    assert prop(lib, ws_bytes=0, aggr=1) == WORKSPACE
    assert prop(lib, ws=None, aggr=1) == WORKSPACE


def test_noalloc_rejects_on_the_host(lib):
    # every argument check of pyg_propagate, then the static scratch limit,
    # all before the device is touched (this runs without a GPU)
    def na(x=FAKE, dtype=0, N=10, F=4, ei=FAKE, E=20, w=None, csr=None, msg=0, aggr=0, kernel=1,
           out=ctypes.c_void_p(0x20000), argmax=None):
        return lib.pyg_propagate_noalloc(x, dtype, N, F, ei, E, w, csr, msg, aggr, kernel, out, argmax, None)
    assert na(dtype=3) == INVALID
    assert na(aggr=2) == INVALID                          # max needs argmax
    assert na(out=ctypes.c_void_p(0x10000 + 8)) == INVALID  # out overlaps x
    assert na(kernel=2) == INVALID                        # CSR kernel needs a CSR
    assert na(N=2**31) == UNSUPPORTED
    # COO max keeps N*F 8-byte keys: 2^20 x 128 needs 1 GiB > the 128 MiB array
    big = 1 << 20
    assert na(N=big, F=128, aggr=2, argmax=ctypes.c_void_p(0x10000000000),
              out=ctypes.c_void_p(0x20000000000), x=ctypes.c_void_p(0x30000000000)) == UNSUPPORTED


def test_other_entry_points_reject_bad_arguments(lib):
    assert lib.pyg_degree(None, 5, 4, FAKE, FAKE, 1 << 30, None) == INVALID
    assert lib.pyg_degree(FAKE, 5, 4, None, FAKE, 1 << 30, None) == INVALID
    assert lib.pyg_degree(FAKE, 5, 2**31, FAKE, FAKE, 1 << 30, None) == UNSUPPORTED
    assert lib.pyg_degree(FAKE, 5, 4, FAKE, FAKE, 0, None) == WORKSPACE
    assert lib.pyg_coo_to_csr(FAKE, 5, 4, None, None, FAKE, FAKE, None, FAKE, 1 << 30, None) == INVALID
    assert lib.pyg_coo_to_csr(FAKE, 5, 4, None, FAKE, FAKE, FAKE, None, FAKE, 0, None) == WORKSPACE
    assert lib.pyg_gcn_norm(FAKE, None, 5, 4, None, FAKE, FAKE, 0, None) == WORKSPACE
    assert lib.pyg_gcn_norm(None, None, 5, 4, None, FAKE, FAKE, 1 << 20, None) == INVALID
    assert lib.pyg_global_pool(FAKE, 0, 10, 4, FAKE, 3, 2, ctypes.c_void_p(0x90000), None, FAKE, 1 << 30, None) == INVALID
    assert lib.pyg_global_pool(FAKE, 0, 10, 4, None, 3, 0, ctypes.c_void_p(0x90000), None, FAKE, 1 << 30, None) == INVALID
    assert lib.pyg_global_pool(FAKE, 0, 10, 4, FAKE, 3, 0, ctypes.c_void_p(0x90000), None, FAKE, 0, None) == WORKSPACE
    assert lib.pyg_global_pool(FAKE, 1, 10, 4, FAKE, 0, 0, ctypes.c_void_p(0x90000), None, FAKE, 1 << 30, None) == INVALID
    assert lib.pyg_validate_coo(None, 5, 4, FAKE, None) == INVALID
    assert lib.pyg_validate_batch(FAKE, 5, 4, None, None) == INVALID


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    import paper_1903_02428_amd.binding as b
    monkeypatch.setattr(b, "_lib", None)
    monkeypatch.setattr(b, "_HERE", str(tmp_path))
    with pytest.raises(b.LibraryMissing):
        b.library()


def test_binding_rejects_host_tensors():
    import torch

    import paper_1903_02428_amd as pyg
    x = torch.zeros(4, 2)
    ei = torch.zeros(2, 3, dtype=torch.int64)
    with pytest.raises(ValueError):
        pyg.propagate(x, ei)
    with pytest.raises(ValueError):
        pyg.degree(ei, 4)


def test_attention_entry_points_reject_bad_arguments(lib):
    from paper_1903_02428_amd.binding import _Csr
    good = _Csr(0x30000, 0x40000, 0x50000, None, 10, 20, 0)
    no_perm = _Csr(0x30000, 0x40000, None, None, 10, 20, 0)
    huge = _Csr(0x30000, 0x40000, 0x50000, None, 10, 2**31, 0)
    A = ctypes.c_void_p(0x90000)
    g = ctypes.byref(good)
    sm = lib.pyg_segment_softmax
    assert sm(FAKE, 2, None, 0, A, FAKE, 1 << 30, None) == INVALID            # no CSR
    assert sm(FAKE, 0, g, 0, A, FAKE, 1 << 30, None) == INVALID               # H = 0
    assert sm(FAKE, 2, g, 5, A, FAKE, 1 << 30, None) == INVALID               # unknown order
    assert sm(FAKE, 2, ctypes.byref(no_perm), 1, A, FAKE, 1 << 30, None) == INVALID  # COO order needs perm
    assert sm(None, 2, g, 0, A, FAKE, 1 << 30, None) == INVALID               # no scores
    assert sm(FAKE, 2, g, 0, None, FAKE, 1 << 30, None) == INVALID            # no output
    assert sm(FAKE, 2, ctypes.byref(huge), 0, A, FAKE, 1 << 30, None) == UNSUPPORTED
    assert sm(FAKE, 2, g, 0, A, FAKE, 0, None) == WORKSPACE
    assert sm(FAKE, 2, g, 0, A, None, 1 << 30, None) == WORKSPACE
    gat = lib.pyg_gat_softmax
    assert gat(FAKE, FAKE, 2, ctypes.c_float(float("nan")), g, 0, A, FAKE, 1 << 30, None) == INVALID
    assert gat(None, FAKE, 2, ctypes.c_float(0.2), g, 0, A, FAKE, 1 << 30, None) == INVALID
    assert gat(FAKE, FAKE, 2, ctypes.c_float(0.2), g, 0, A, FAKE, 0, None) == WORKSPACE
    bwd = lib.pyg_segment_softmax_backward
    assert bwd(FAKE, None, 2, g, 0, A, FAKE, 1 << 30, None) == INVALID
    assert bwd(FAKE, FAKE, 2, g, 0, A, FAKE, 0, None) == WORKSPACE
    ph = lib.pyg_propagate_heads
    X, OUT = FAKE, ctypes.c_void_p(0x200000)
    assert ph(X, 0, 10, 0, 4, g, A, OUT, FAKE, 1 << 30, None) == INVALID       # H = 0
    assert ph(X, 0, 11, 2, 4, g, A, OUT, FAKE, 1 << 30, None) == INVALID       # CSR of another graph
    assert ph(X, 0, 10, 2, 4, g, None, OUT, FAKE, 1 << 30, None) == INVALID    # no alpha
    assert ph(X, 0, 10, 2, 4, None, A, OUT, FAKE, 1 << 30, None) == INVALID    # no CSR
    assert ph(X, 3, 10, 2, 4, g, A, OUT, FAKE, 1 << 30, None) == INVALID       # bad dtype
    assert ph(X, 0, 10, 2, 4, g, A, ctypes.c_void_p(0x10000 + 16), FAKE, 1 << 30, None) == INVALID  # out overlaps x
    assert ph(X, 0, 10, 2, 4, g, A, OUT, FAKE, 0, None) == WORKSPACE
    last = 0
    for E in (0, 100, 10**5, 10**7):
        rc, b = _ws(lib.pyg_segment_softmax_workspace, E, 1000, 4, 0)
        assert rc == PYG_OK and b >= last
        last = b
    assert _ws(lib.pyg_segment_softmax_workspace, 10, 5, -1, 0)[0] == INVALID
    assert _ws(lib.pyg_propagate_heads_workspace, 0, 10, 2, 4, 20, 0)[0] == PYG_OK
    assert _ws(lib.pyg_propagate_heads_workspace, 0, 10, 2**20, 2**12, 20, 0)[0] == UNSUPPORTED


def test_dense_transform_rejects_bad_arguments(lib):
    X, T, OUT = FAKE, ctypes.c_void_p(0x300000), ctypes.c_void_p(0x900000)
    dt = lib.pyg_dense_transform
    assert dt(X, 0, 10, 8, T, 4, OUT, 0, FAKE, 0, None) == WORKSPACE   # fp32 operands: accepted, checked further
    assert dt(X, 0, 10, 8, T, 4, ctypes.c_void_p(0x10000 + 64), 0, FAKE, 1 << 30, None) == INVALID  # overlap (4-byte x)
    assert dt(X, 7, 10, 8, T, 4, OUT, 0, FAKE, 1 << 30, None) == INVALID       # bad dtype
    assert dt(X, 1, 10, 8, T, 4, OUT, 9, FAKE, 1 << 30, None) == INVALID       # bad out dtype
    assert dt(X, 1, -1, 8, T, 4, OUT, 0, FAKE, 1 << 30, None) == INVALID
    assert dt(None, 1, 10, 8, T, 4, OUT, 0, FAKE, 1 << 30, None) == INVALID
    assert dt(X, 1, 10, 8, None, 4, OUT, 0, FAKE, 1 << 30, None) == INVALID
    assert dt(X, 1, 10, 8, T, 4, None, 0, FAKE, 1 << 30, None) == INVALID
    assert dt(X, 1, 10, 8, T, 4, OUT, 0, FAKE, 0, None) == WORKSPACE
    assert dt(X, 1, 10, 8, T, 4, ctypes.c_void_p(0x10000 + 32), 0, FAKE, 1 << 30, None) == INVALID  # overlap
    assert dt(X, 1, 2**31, 8, T, 4, OUT, 0, FAKE, 1 << 30, None) == UNSUPPORTED
    rc, b = _ws(lib.pyg_dense_transform_workspace, 602, 41)
    assert rc == PYG_OK and b >= 48 * 608 * 2 and b >= 48 * 608 * 4  # bf16 or fp32 Theta^T


def test_propagate_edge_rejects_bad_arguments(lib):
    from paper_1903_02428_amd.binding import _Csr
    EA, OUT = ctypes.c_void_p(0x500000), ctypes.c_void_p(0x900000)
    good = _Csr(0x30000, 0x40000, 0x50000, None, 10, 20, 0)
    no_perm = _Csr(0x30000, 0x40000, None, None, 10, 20, 0)

    def pe(x=FAKE, dtype=0, N=10, F=4, ei=FAKE, E=20, ea=EA, order=1, csr=None, msg=2, aggr=0, kernel=1, out=OUT,
           argmax=None, ws=FAKE, ws_bytes=1 << 40):
        return lib.pyg_propagate_edge(x, dtype, N, F, ei, E, ea, order, csr, msg, aggr, kernel, out, argmax, ws,
                                      ws_bytes, None)
    assert pe(msg=0) == INVALID                          # plain messages go through pyg_propagate
    assert pe(msg=1) == INVALID
    assert pe(msg=5) == INVALID
    assert pe(order=3) == INVALID
    assert pe(ea=None) == INVALID                        # edge messages need the features
    assert pe(order=0) == INVALID                        # the COO kernel reads edges in COO order
    assert pe(aggr=2) == INVALID                         # max needs argmax
    assert pe(ei=None) == INVALID                        # COO kernel needs edges
    assert pe(kernel=2, csr=ctypes.byref(no_perm), order=1) == INVALID  # COO-ordered features need perm
    assert pe(kernel=2, csr=None) == INVALID
    assert pe(out=ctypes.c_void_p(0x500000 + 64)) == INVALID  # out overlaps the edge features
    assert pe(N=2**31) == UNSUPPORTED
    assert pe(kernel=2, csr=ctypes.byref(good), order=0, ws_bytes=0) == WORKSPACE
    assert pe(ws_bytes=0, aggr=1) == WORKSPACE


def test_attention_backward_rejects_bad_arguments(lib):
    from paper_1903_02428_amd.binding import _Csr
    good = ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 10, 20, 0))
    other = ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 11, 20, 0))
    no_perm = ctypes.byref(_Csr(0x30000, 0x40000, None, None, 10, 20, 0))
    G, X, A, GX, GA = FAKE, ctypes.c_void_p(0x200000), ctypes.c_void_p(0x300000), ctypes.c_void_p(0x400000), \
        ctypes.c_void_p(0x500000)
    hb = lib.pyg_propagate_heads_backward
    assert hb(G, X, 0, 10, 2, 4, good, None, None, A, GX, GA, FAKE, 1 << 30, None) == INVALID   # no reversed CSR
    assert hb(G, X, 0, 10, 2, 4, good, other, None, A, GX, GA, FAKE, 1 << 30, None) == INVALID  # other graphs
    assert hb(G, X, 0, 10, 2, 4, good, no_perm, None, A, GX, GA, FAKE, 1 << 30, None) == INVALID
    assert hb(G, X, 0, 10, 0, 4, good, good, None, A, GX, GA, FAKE, 1 << 30, None) == INVALID    # H = 0
    assert hb(G, X, 0, 10, 2, 4, good, good, None, None, GX, GA, FAKE, 1 << 30, None) == INVALID  # no alpha
    assert hb(G, None, 0, 10, 2, 4, good, good, None, A, GX, GA, FAKE, 1 << 30, None) == INVALID  # grad_alpha needs x
    assert hb(G, X, 0, 10, 2, 4, good, good, None, A, None, None, FAKE, 1 << 30, None) == INVALID  # nothing to do
    assert hb(G, X, 0, 10, 2, 4, good, good, None, A, GX, GA, FAKE, 0, None) == WORKSPACE
    gb = lib.pyg_gat_scores_backward
    inf = ctypes.c_float(float("inf"))
    assert gb(A, A, 2, inf, good, good, None, G, GX, GA, FAKE, 1 << 30, None) == INVALID
    assert gb(A, A, 2, ctypes.c_float(0.2), good, None, None, G, GX, GA, FAKE, 1 << 30, None) == INVALID
    assert gb(A, A, 2, ctypes.c_float(0.2), good, good, None, None, GX, GA, FAKE, 1 << 30, None) == INVALID
    assert gb(A, A, 2, ctypes.c_float(0.2), good, good, None, G, GX, GA, FAKE, 0, None) == WORKSPACE
    tm = lib.pyg_csr_transpose_map
    assert tm(good, None, FAKE, FAKE, 1 << 30, None) == INVALID
    assert tm(good, other, FAKE, FAKE, 1 << 30, None) == INVALID
    assert tm(good, no_perm, FAKE, FAKE, 1 << 30, None) == INVALID
    assert tm(good, good, None, FAKE, 1 << 30, None) == INVALID  # no output
    assert tm(good, good, FAKE, FAKE, 0, None) == WORKSPACE


def test_degree_csr_rejects_bad_arguments(lib):
    from paper_1903_02428_amd.binding import _Csr
    assert lib.pyg_degree_csr(None, FAKE, None) == INVALID
    assert lib.pyg_degree_csr(ctypes.byref(_Csr(None, 0x40000, 0x50000, None, 10, 20, 0)), FAKE, None) == INVALID
    assert lib.pyg_degree_csr(ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 10, 20, 0)), None, None) == INVALID
    assert lib.pyg_degree_csr(ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 0, 0, 0)), None, None) == 0  # N = 0


def test_edge_backward_rejects_bad_arguments(lib):
    from paper_1903_02428_amd.binding import _Csr
    good = ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 10, 20, 0))
    other = ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 11, 20, 0))
    G, X, EA, GX, GE = FAKE, ctypes.c_void_p(0x200000), ctypes.c_void_p(0x300000), ctypes.c_void_p(0x400000), \
        ctypes.c_void_p(0x500000)
    eb = lib.pyg_propagate_edge_backward
    RELU, ADD, SUM, MAX = 3, 2, 0, 2
    assert eb(G, X, EA, 2, 10, 4, FAKE, good, good, None, 0, RELU, SUM, None, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, FAKE, good, good, None, 0, 0, SUM, None, GX, GE, FAKE, 1 << 30, None) == INVALID  # msg
    assert eb(G, X, EA, 0, 10, 4, FAKE, good, good, None, 2, RELU, SUM, None, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, FAKE, None, good, None, 0, RELU, SUM, None, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, FAKE, good, None, None, 0, RELU, SUM, None, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, FAKE, good, other, None, 0, RELU, SUM, None, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, None, EA, 0, 10, 4, FAKE, good, good, None, 0, RELU, SUM, None, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, FAKE, good, good, None, 0, RELU, SUM, None, None, None, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, None, good, good, None, 0, RELU, MAX, FAKE, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, FAKE, good, good, None, 0, RELU, MAX, None, GX, GE, FAKE, 1 << 30, None) == INVALID
    assert eb(G, X, EA, 0, 10, 4, FAKE, good, good, None, 0, ADD, SUM, None, GX, GE, FAKE, 0, None) == WORKSPACE


def test_edge_backward_workspace_sizes(lib):
    """bf16 adds only fp32 scratch: none under sum, grad_x's N*F*4 under
    max and mean, and under mean with relu / mul also x and the edge rows
    widened (N*F*4 + E*F*4). Sizes here are multiples of the 256-byte carve
    alignment, so the differences are exact."""
    ws = lib.pyg_propagate_edge_backward_workspace
    N, F, E = 1000, 16, 5000
    ADD, RELU, MUL, SUM, MEAN, MAX = 2, 3, 4, 0, 1, 2

    def q(dt, msg, aggr, chunk=0):
        sz = ctypes.c_size_t()
        assert ws(dt, N, F, E, msg, aggr, chunk, ctypes.byref(sz)) == 0
        return sz.value

    for msg in (ADD, RELU, MUL):
        assert q(1, msg, SUM) == q(0, msg, SUM)
        assert q(1, msg, MAX) == q(0, msg, MAX) + N * F * 4
    assert q(1, ADD, MEAN) == q(0, ADD, MEAN) + N * F * 4
    for msg in (RELU, MUL):
        assert q(1, msg, MEAN) == q(0, msg, MEAN) + 2 * N * F * 4 + E * F * 4
    sz = ctypes.c_size_t()
    assert ws(2, N, F, E, RELU, SUM, 0, ctypes.byref(sz)) == INVALID  # dtype
    assert ws(0, N, F, E, 0, SUM, 0, ctypes.byref(sz)) == INVALID  # not an edge-feature message
    assert ws(0, N, F, E, RELU, 3, 0, ctypes.byref(sz)) == INVALID
    assert ws(0, N, F, E, RELU, SUM, 0, None) == INVALID
    assert ws(0, N, F, 1 << 31, RELU, SUM, 0, ctypes.byref(sz)) == -5


def test_backward_rejects_bad_grad_w_order(lib):
    from paper_1903_02428_amd.binding import _Csr
    good = ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, 0x60000, 10, 20, 0))
    G, X, GX, GW = FAKE, ctypes.c_void_p(0x200000), ctypes.c_void_p(0x400000), ctypes.c_void_p(0x500000)
    bw = lib.pyg_propagate_backward
    SUM, MAX, CSR, COO = 0, 2, 0, 1
    assert bw(G, X, 0, 10, 4, FAKE, 20, FAKE, good, good, 0, SUM, None, GX, GW, 7, FAKE, 1 << 30, None) == INVALID
    # max with grad_w in CSR order needs the forward CSR (its perm maps edge ids to slots)
    assert bw(G, X, 0, 10, 4, FAKE, 20, FAKE, None, None, 0, MAX, FAKE, GX, GW, CSR, FAKE, 1 << 30, None) == INVALID
    assert bw(G, X, 0, 10, 4, FAKE, 20, FAKE, None, None, 0, MAX, FAKE, GX, GW, COO, FAKE, 0, None) == WORKSPACE


def test_edge_encoded_rejects_bad_arguments(lib):
    from paper_1903_02428_amd.binding import _Csr
    good = ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 10, 20, 0))
    X, EA, TH, OUT = FAKE, ctypes.c_void_p(0x300000), ctypes.c_void_p(0x400000), ctypes.c_void_p(0x900000)
    en = lib.pyg_propagate_edge_encoded
    ADD, SUM, CSRK = 2, 0, 2
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, TH, 0, good, 0, SUM, CSRK, OUT, None, FAKE, 1 << 30, None) == INVALID  # msg
    assert en(X, 0, 10, 4, FAKE, 20, None, 3, TH, 0, good, ADD, SUM, CSRK, OUT, None, FAKE, 1 << 30, None) == INVALID
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, None, 0, good, ADD, SUM, CSRK, OUT, None, FAKE, 1 << 30, None) == INVALID
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, TH, 0, None, ADD, SUM, CSRK, OUT, None, FAKE, 1 << 30, None) == INVALID
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, TH, 0, good, ADD, SUM, CSRK, OUT, None, FAKE, 0, None) == WORKSPACE
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, TH, 0, good, ADD, SUM, CSRK, FAKE, None, FAKE, 1 << 30, None) == INVALID
    WS = ctypes.c_void_p(0x1000000)
    assert en(ctypes.c_void_p(0x1000040), 0, 10, 4, FAKE, 20, EA, 3, TH, 0, good, ADD, SUM, CSRK, OUT, None, WS,
              1 << 20, None) == INVALID  # x inside the workspace
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, ctypes.c_void_p(0x1000040), 0, good, ADD, SUM, CSRK, OUT, None, WS,
              1 << 20, None) == INVALID  # theta_e inside the workspace
    # every check of the edge propagate comes before the projection runs
    other = ctypes.byref(_Csr(0x30000, 0x40000, 0x50000, None, 11, 20, 0))
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, TH, 0, other, ADD, SUM, CSRK, OUT, None, FAKE, 1 << 30, None) == INVALID
    assert en(X, 0, 0, 4, FAKE, 20, EA, 3, TH, 0, None, ADD, SUM, 1, OUT, None, FAKE, 1 << 30, None) == INVALID
    assert en(X, 0, 10, 4, FAKE, 20, EA, 3, TH, 1, good, ADD, 2, CSRK, OUT, None, FAKE, 1 << 30, None) == INVALID
    rc, b = _ws(lib.pyg_propagate_edge_encoded_workspace, 0, 10, 4, 20, 3, SUM, CSRK, 0)
    assert rc == PYG_OK and b >= 20 * 4 * 4
