"""ctypes binding of libpyg_mi355x.so (argument marshalling only)."""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch  # loads the HIP runtime the library must share, before the library itself

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_NAME = "libpyg_mi355x.so"

PYG_OK = 0
DTYPE = {torch.float32: 0, torch.bfloat16: 1}
AGGR = {"sum": 0, "mean": 1, "max": 2}
MSG = {"src": 0, "diff": 1, "edge_add": 2, "edge_relu": 3, "edge_mul": 4}
KERNEL = {"auto": 0, "coo": 1, "csr": 2}
ORDER = {"csr": 0, "coo": 1}

EXPORTED = [
    "pyg_strerror", "pyg_abi_version", "pyg_degree_workspace", "pyg_degree", "pyg_degree_csr",
    "pyg_coo_to_csr_workspace",
    "pyg_coo_to_csr", "pyg_gather_edges",
    "pyg_gcn_norm_workspace", "pyg_gcn_norm", "pyg_gcn_norm_csr_workspace", "pyg_gcn_norm_csr",
    "pyg_propagate_workspace", "pyg_propagate", "pyg_propagate_edge", "pyg_propagate_edge_encoded_workspace",
    "pyg_propagate_edge_encoded", "pyg_propagate_backward_workspace",
    "pyg_propagate_backward", "pyg_propagate_edge_backward_workspace", "pyg_propagate_edge_backward",
    "pyg_segment_softmax_workspace", "pyg_segment_softmax", "pyg_gat_softmax", "pyg_segment_softmax_backward",
    "pyg_propagate_heads_workspace", "pyg_propagate_heads", "pyg_dense_transform_workspace", "pyg_dense_transform",
    "pyg_csr_transpose_map_workspace", "pyg_csr_transpose_map",
    "pyg_propagate_heads_backward_workspace", "pyg_propagate_heads_backward", "pyg_gat_scores_backward_workspace",
    "pyg_gat_scores_backward",
    "pyg_global_pool_workspace", "pyg_global_pool", "pyg_validate_coo", "pyg_validate_batch",
    "pyg_propagate_noalloc", "pyg_gcn_propagate_workspace", "pyg_gcn_propagate", "pyg_csr_blocks_workspace", "pyg_csr_blocks_build", "pyg_propagate_blocked_workspace",
    "pyg_propagate_blocked", "pyg_gcn_propagate_blocked_workspace", "pyg_gcn_propagate_blocked",
    "pyg_coo_to_csr_blocked_workspace", "pyg_coo_to_csr_blocked", "pyg_degree_csr_blocks",
]


class LibraryMissing(RuntimeError):
    """The HIP library has not been built (run __graft_entry__.build())."""


class PygError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {strerror(status)} (status {status})")
        self.status = status


class _Csr(ctypes.Structure):
    _fields_ = [("rowptr", ctypes.c_void_p), ("col", ctypes.c_void_p), ("perm", ctypes.c_void_p),
                ("weight", ctypes.c_void_p), ("N", ctypes.c_int64), ("E", ctypes.c_int64),
                ("chunk", ctypes.c_int64)]


class _CsrBlocks(ctypes.Structure):
    _fields_ = [("rowptr", ctypes.c_void_p), ("col", ctypes.c_void_p), ("perm", ctypes.c_void_p),
                ("weight", ctypes.c_void_p), ("N", ctypes.c_int64), ("E", ctypes.c_int64), ("B", ctypes.c_int64),
                ("chunk", ctypes.c_int64)]


_lib = None


def library_path() -> str:
    return os.path.join(_HERE, LIB_NAME)


def library() -> ctypes.CDLL:
    """Load the library (once). Raises LibraryMissing if it was never built."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise LibraryMissing(f"{path} not found: build it with paper_1903_02428_amd.build.build()")
        lib = ctypes.CDLL(path)
        p, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)
        lib.pyg_strerror.argtypes, lib.pyg_strerror.restype = [i32], ctypes.c_char_p
        lib.pyg_abi_version.argtypes, lib.pyg_abi_version.restype = [], i32
        sigs = {
            "pyg_degree_workspace": [i64, i64, sz],
            "pyg_degree": [p, i64, i64, p, p, ctypes.c_size_t, p],
            "pyg_degree_csr": [ctypes.POINTER(_Csr), p, p],
            "pyg_coo_to_csr_workspace": [i64, i64, sz],
            "pyg_coo_to_csr": [p, i64, i64, p, p, p, p, p, p, ctypes.c_size_t, p],
            "pyg_gather_edges": [p, i64, p, p, p],
            "pyg_gcn_norm_workspace": [i64, i64, sz],
            "pyg_gcn_norm": [p, p, i64, i64, p, p, p, ctypes.c_size_t, p],
            "pyg_gcn_norm_csr_workspace": [i64, sz],
            "pyg_gcn_norm_csr": [ctypes.POINTER(_Csr), p, p, ctypes.c_size_t, p],
            "pyg_propagate_workspace": [i32, i64, i64, i64, i32, i32, i64, sz],
            "pyg_propagate": [p, i32, i64, i64, p, i64, p, ctypes.POINTER(_Csr), i32, i32, i32, p, p, p,
                              ctypes.c_size_t, p],
            "pyg_gcn_propagate_workspace": [i32, i64, i64, i64, i64, sz],
            "pyg_gcn_propagate": [p, i32, i64, i64, ctypes.POINTER(_Csr), p, p, p, ctypes.c_size_t, p],
            "pyg_csr_blocks_workspace": [i64, i64, i64, sz],
            "pyg_csr_blocks_build": [ctypes.POINTER(_Csr), i64, p, p, p, p, p, ctypes.c_size_t, p],
            "pyg_propagate_blocked_workspace": [i32, i64, i64, i64, i64, i32, i64, sz],
            "pyg_gcn_propagate_blocked_workspace": [i32, i64, i64, i64, i64, i64, sz],
            "pyg_coo_to_csr_blocked_workspace": [i64, i64, i64, sz],
            "pyg_coo_to_csr_blocked": [p, i64, i64, i64, p, p, p, p, p, p, ctypes.c_size_t, p],
            "pyg_degree_csr_blocks": [ctypes.POINTER(_CsrBlocks), p, p],
            "pyg_gcn_propagate_blocked": [p, i32, i64, i64, ctypes.POINTER(_Csr), ctypes.POINTER(_CsrBlocks), p, p, p,
                                          ctypes.c_size_t, p],
            "pyg_propagate_blocked": [p, i32, i64, i64, ctypes.POINTER(_CsrBlocks), i32, i32, p, p, p, ctypes.c_size_t,
                                      p],
            "pyg_propagate_noalloc": [p, i32, i64, i64, p, i64, p, ctypes.POINTER(_Csr), i32, i32, i32, p, p, p],
            "pyg_propagate_edge": [p, i32, i64, i64, p, i64, p, i32, ctypes.POINTER(_Csr), i32, i32, i32, p, p, p,
                                   ctypes.c_size_t, p],
            "pyg_propagate_edge_encoded_workspace": [i32, i64, i64, i64, i64, i32, i32, i64, sz],
            "pyg_propagate_edge_encoded": [p, i32, i64, i64, p, i64, p, i64, p, i32, ctypes.POINTER(_Csr), i32, i32,
                                           i32, p, p, p, ctypes.c_size_t, p],
            "pyg_propagate_backward_workspace": [i32, i64, i64, i64, i32, i64, sz],
            "pyg_propagate_backward": [p, p, i32, i64, i64, p, i64, p, ctypes.POINTER(_Csr), ctypes.POINTER(_Csr),
                                       i32, i32, p, p, p, i32, p, ctypes.c_size_t, p],
            "pyg_propagate_edge_backward_workspace": [i32, i64, i64, i64, i32, i32, i64, sz],
            "pyg_propagate_edge_backward": [p, p, p, i32, i64, i64, p, ctypes.POINTER(_Csr), ctypes.POINTER(_Csr), p,
                                            i32, i32, i32, p, p, p, p, ctypes.c_size_t, p],
            "pyg_segment_softmax_workspace": [i64, i64, i64, i64, sz],
            "pyg_segment_softmax": [p, i64, ctypes.POINTER(_Csr), i32, p, p, ctypes.c_size_t, p],
            "pyg_gat_softmax": [p, p, i64, ctypes.c_float, ctypes.POINTER(_Csr), i32, p, p, ctypes.c_size_t, p],
            "pyg_segment_softmax_backward": [p, p, i64, ctypes.POINTER(_Csr), i32, p, p, ctypes.c_size_t, p],
            "pyg_propagate_heads_workspace": [i32, i64, i64, i64, i64, i64, sz],
            "pyg_propagate_heads": [p, i32, i64, i64, i64, ctypes.POINTER(_Csr), p, p, p, ctypes.c_size_t, p],
            "pyg_dense_transform_workspace": [i64, i64, sz],
            "pyg_propagate_heads_backward_workspace": [i32, i64, i64, i64, i64, i64, sz],
            "pyg_csr_transpose_map_workspace": [i64, sz],
            "pyg_csr_transpose_map": [ctypes.POINTER(_Csr), ctypes.POINTER(_Csr), p, p, ctypes.c_size_t, p],
            "pyg_propagate_heads_backward": [p, p, i32, i64, i64, i64, ctypes.POINTER(_Csr), ctypes.POINTER(_Csr), p, p,
                                             p, p, p, ctypes.c_size_t, p],
            "pyg_gat_scores_backward_workspace": [i64, i64, i64, i64, sz],
            "pyg_gat_scores_backward": [p, p, i64, ctypes.c_float, ctypes.POINTER(_Csr), ctypes.POINTER(_Csr), p, p, p,
                                        p, p, ctypes.c_size_t, p],
            "pyg_dense_transform": [p, i32, i64, i64, p, i64, p, i32, p, ctypes.c_size_t, p],
            "pyg_global_pool_workspace": [i32, i64, i64, i64, i32, sz],
            "pyg_global_pool": [p, i32, i64, i64, p, i64, i32, p, p, p, ctypes.c_size_t, p],
            "pyg_validate_coo": [p, i64, i64, p, p],
            "pyg_validate_batch": [p, i64, i64, p, p],
        }
        for name, args in sigs.items():
            fn = getattr(lib, name)
            fn.argtypes, fn.restype = args, i32
        _lib = lib
    return _lib


def strerror(status: int) -> str:
    return library().pyg_strerror(int(status)).decode()


def abi_version() -> int:
    return int(library().pyg_abi_version())


def _check(rc: int, what: str):
    if rc != PYG_OK:
        raise PygError(rc, what)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need_cuda(name, t, dtype=None, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a HIP device, got {t.device}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _edge_index(edge_index):
    _need_cuda("edge_index", edge_index, torch.int64, 2)
    if edge_index.shape[0] != 2:
        raise ValueError("edge_index must be [2, E]")
    return edge_index.shape[1]


def _workspace(nbytes: int, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _size(fn, *args) -> int:
    out = ctypes.c_size_t(0)
    _check(fn(*args, ctypes.byref(out)), fn.__name__)
    return int(out.value)


@dataclass
class CSR:
    """Target-sorted CSR built on the device by pyg_coo_to_csr."""
    rowptr: torch.Tensor   # int64 [N+1]
    col: torch.Tensor      # int32 [E]
    perm: torch.Tensor     # int64 [E]
    weight: torch.Tensor | None  # fp32 [E] CSR order
    N: int
    E: int
    chunk: int = 0

    def _c(self) -> _Csr:
        return _Csr(self.rowptr.data_ptr(), self.col.data_ptr() if self.E else None,
                    self.perm.data_ptr() if self.E else None,
                    None if self.weight is None else self.weight.data_ptr(), self.N, self.E, self.chunk)


@dataclass
class CSRBlocks:
    """A CSR regrouped by source block (pyg_csr_blocks_build): virtual row
    b * N + i holds the slots of target i whose source lies in block b."""
    rowptr: torch.Tensor         # int64 [B*N+1]
    col: torch.Tensor            # int32 [E]
    perm: torch.Tensor | None    # int64 [E] COO edge ids, or None
    weight: torch.Tensor | None  # fp32 [E] in this slot order, or None
    N: int
    E: int
    B: int
    chunk: int = 0

    def _c(self) -> _CsrBlocks:
        return _CsrBlocks(self.rowptr.data_ptr(), self.col.data_ptr() if self.E else None,
                          None if self.perm is None or not self.E else self.perm.data_ptr(),
                          None if self.weight is None or not self.E else self.weight.data_ptr(),
                          self.N, self.E, self.B, self.chunk)


def csr_blocks(csr: CSR, B: int = 8, with_perm: bool = False, with_weight: bool | None = None,
               out: CSRBlocks | None = None, workspace: torch.Tensor | None = None) -> CSRBlocks:
    """Regroup a CSR's slots by source block (2 <= B <= 32). The
    weights come along when the CSR has them (unless with_weight is False);
    the edge ids (needed for max) when with_perm."""
    lib = library()
    dev = csr.rowptr.device
    with_weight = csr.weight is not None if with_weight is None else with_weight
    if with_weight and csr.weight is None:
        raise ValueError("the CSR has no weights")
    if out is not None:
        if out.N != csr.N or out.E != csr.E or out.B != B or (out.perm is None) == with_perm or \
                (out.weight is None) == with_weight:
            raise ValueError("out CSRBlocks has another shape")
        rowptr, col, perm, w = out.rowptr, out.col, out.perm, out.weight
    else:
        rowptr = torch.empty(B * csr.N + 1, dtype=torch.int64, device=dev)
        col = torch.empty(csr.E, dtype=torch.int32, device=dev)
        perm = torch.empty(csr.E, dtype=torch.int64, device=dev) if with_perm else None
        w = torch.empty(csr.E, dtype=torch.float32, device=dev) if with_weight else None
    nbytes = _size(lib.pyg_csr_blocks_workspace, csr.N, csr.E, B)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    c = csr._c()
    _check(lib.pyg_csr_blocks_build(ctypes.byref(c), B, _ptr(rowptr), _ptr(col), _ptr(perm), _ptr(w), _ptr(ws), nbytes,
                                    _stream(dev)), "pyg_csr_blocks_build")
    if out is not None:
        out.chunk = csr.chunk
        return out
    return CSRBlocks(rowptr, col, perm, w, csr.N, csr.E, B, csr.chunk)


def propagate_blocked_workspace_bytes(x: torch.Tensor, bcsr: CSRBlocks, aggr: str) -> int:
    return _size(library().pyg_propagate_blocked_workspace, DTYPE[x.dtype], x.shape[0], x.shape[1], bcsr.E, bcsr.B,
                 AGGR[aggr], bcsr.chunk)


def propagate_blocked(x: torch.Tensor, bcsr: CSRBlocks, aggr: str = "sum", msg: str = "src",
                      out: torch.Tensor | None = None, argmax: torch.Tensor | None = None,
                      workspace: torch.Tensor | None = None):
    """Eq. (1) over a source-blocked CSR (pyg_propagate_blocked): the same
    results as propagate() with the CSR kernel. Returns (out, argmax or None)."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    if bcsr.N != N:
        raise ValueError("bcsr does not match x")
    if aggr not in AGGR or msg not in ("src", "diff"):
        raise ValueError("bad aggr / msg")
    if out is None:
        out = torch.empty_like(x)
    if aggr == "max" and argmax is None:
        argmax = torch.empty((N, F), dtype=torch.int64, device=x.device)
    if aggr != "max":
        argmax = None
    nbytes = propagate_blocked_workspace_bytes(x, bcsr, aggr)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, x.device)
    c = bcsr._c()
    rc = lib.pyg_propagate_blocked(_ptr(x), DTYPE[x.dtype], N, F, ctypes.byref(c), MSG[msg], AGGR[aggr], _ptr(out),
                                   _ptr(argmax), _ptr(workspace), workspace.numel(), _stream(x.device))
    _check(rc, "pyg_propagate_blocked")
    return out, argmax


def degree(edge_index: torch.Tensor, num_nodes: int, out: torch.Tensor | None = None,
           workspace: torch.Tensor | None = None) -> torch.Tensor:
    lib = library()
    E = _edge_index(edge_index)
    dev = edge_index.device
    deg = torch.empty(num_nodes, dtype=torch.int64, device=dev) if out is None else out
    nbytes = _size(lib.pyg_degree_workspace, E, num_nodes)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    _check(lib.pyg_degree(_ptr(edge_index), E, num_nodes, _ptr(deg), _ptr(ws), ws.numel(), _stream(dev)),
           "pyg_degree")
    return deg


def degree_csr(csr: "CSR", out: torch.Tensor | None = None) -> torch.Tensor:
    """In-degree read off a CSR's row boundaries (the same counts as
    degree() on the edge list the CSR was built from)."""
    lib = library()
    dev = csr.rowptr.device
    if out is None:
        out = torch.empty(csr.N, dtype=torch.int64, device=dev)
    else:
        _need_cuda("out", out, torch.int64, 1)
        if out.shape[0] != csr.N:
            raise ValueError("out must be [N]")
    c = csr._c()
    _check(lib.pyg_degree_csr(ctypes.byref(c), _ptr(out), _stream(dev)), "pyg_degree_csr")
    return out


def coo_to_csr(edge_index: torch.Tensor, num_nodes: int, edge_weight: torch.Tensor | None = None,
               chunk: int = 0, out: CSR | None = None, workspace: torch.Tensor | None = None) -> CSR:
    """Build the CSR; `out` (a CSR of the same shape) and `workspace` may be
    passed to reuse device buffers."""
    lib = library()
    E = _edge_index(edge_index)
    dev = edge_index.device
    if edge_weight is not None:
        _need_cuda("edge_weight", edge_weight, torch.float32, 1)
        if edge_weight.shape[0] != E:
            raise ValueError("edge_weight must be [E]")
    if out is not None:
        if out.N != num_nodes or out.E != E or ((out.weight is None) != (edge_weight is None)):
            raise ValueError("out CSR has another shape")
        rowptr, col, perm, wcsr = out.rowptr, out.col, out.perm, out.weight
    else:
        rowptr = torch.empty(num_nodes + 1, dtype=torch.int64, device=dev)
        col = torch.empty(E, dtype=torch.int32, device=dev)
        perm = torch.empty(E, dtype=torch.int64, device=dev)
        wcsr = torch.empty(E, dtype=torch.float32, device=dev) if edge_weight is not None else None
    nbytes = _size(lib.pyg_coo_to_csr_workspace, E, num_nodes)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    _check(lib.pyg_coo_to_csr(_ptr(edge_index), E, num_nodes, _ptr(edge_weight), _ptr(rowptr), _ptr(col),
                              _ptr(perm), _ptr(wcsr), _ptr(ws), nbytes, _stream(dev)), "pyg_coo_to_csr")
    if out is not None:
        out.chunk = chunk
        return out
    return CSR(rowptr, col, perm, wcsr, num_nodes, E, chunk)


def coo_to_csr_blocked(edge_index: torch.Tensor, num_nodes: int, B: int, edge_weight: torch.Tensor | None = None,
                       with_perm: bool = False, chunk: int = 0, out: "CSRBlocks | None" = None,
                       workspace: torch.Tensor | None = None) -> "CSRBlocks":
    """The source-blocked CSR straight from the COO (pyg_coo_to_csr_blocked):
    the same arrays as csr_blocks(coo_to_csr(...), B), in one sort. The edge
    ids (needed for max) when with_perm; `out` and `workspace` may be passed
    to reuse device buffers."""
    lib = library()
    E = _edge_index(edge_index)
    dev = edge_index.device
    if edge_weight is not None:
        _need_cuda("edge_weight", edge_weight, torch.float32, 1)
        if edge_weight.shape[0] != E:
            raise ValueError("edge_weight must be [E]")
    if out is not None:
        if out.N != num_nodes or out.E != E or out.B != B or (out.perm is None) == with_perm or \
                ((out.weight is None) != (edge_weight is None)):
            raise ValueError("out CSRBlocks has another shape")
        rowptr, col, perm, wcsr = out.rowptr, out.col, out.perm, out.weight
    else:
        rowptr = torch.empty(B * num_nodes + 1, dtype=torch.int64, device=dev)
        col = torch.empty(E, dtype=torch.int32, device=dev)
        perm = torch.empty(E, dtype=torch.int64, device=dev) if with_perm else None
        wcsr = torch.empty(E, dtype=torch.float32, device=dev) if edge_weight is not None else None
    nbytes = _size(lib.pyg_coo_to_csr_blocked_workspace, E, num_nodes, B)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    _check(lib.pyg_coo_to_csr_blocked(_ptr(edge_index), E, num_nodes, B, _ptr(edge_weight), _ptr(rowptr), _ptr(col),
                                      _ptr(perm), _ptr(wcsr), _ptr(ws), nbytes, _stream(dev)),
           "pyg_coo_to_csr_blocked")
    if out is not None:
        out.chunk = chunk
        return out
    return CSRBlocks(rowptr, col, perm, wcsr, num_nodes, E, B, chunk)


def coo_to_csr_blocked_workspace_bytes(E: int, num_nodes: int, B: int) -> int:
    return _size(library().pyg_coo_to_csr_blocked_workspace, E, num_nodes, B)


def degree_csr_blocks(bcsr: "CSRBlocks", out: torch.Tensor | None = None) -> torch.Tensor:
    """In-degree from a source-blocked CSR (the slots of each target over all
    blocks; the same counts as degree())."""
    lib = library()
    dev = bcsr.rowptr.device
    if out is None:
        out = torch.empty(bcsr.N, dtype=torch.int64, device=dev)
    else:
        _need_cuda("out", out, torch.int64, 1)
        if out.shape[0] != bcsr.N:
            raise ValueError("out must be [N]")
    c = bcsr._c()
    _check(lib.pyg_degree_csr_blocks(ctypes.byref(c), _ptr(out), _stream(dev)), "pyg_degree_csr_blocks")
    return out


def gather_edges(perm: torch.Tensor, values: torch.Tensor) -> torch.Tensor:
    """values[perm] for a COO-ordered fp32 edge array (CSR slot order out)."""
    _need_cuda("perm", perm, torch.int64, 1)
    _need_cuda("values", values, torch.float32, 1)
    if values.shape != perm.shape:
        raise ValueError("perm and values must both be [E]")
    out = torch.empty_like(values)
    _check(library().pyg_gather_edges(_ptr(perm), perm.shape[0], _ptr(values), _ptr(out), _stream(perm.device)),
           "pyg_gather_edges")
    return out


def gcn_norm(edge_index: torch.Tensor, num_nodes: int, edge_weight: torch.Tensor | None = None,
             out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
             deg: torch.Tensor | None = None) -> torch.Tensor:
    """GCN edge norms; `deg` may pass the in-degree already computed by degree()."""
    lib = library()
    E = _edge_index(edge_index)
    dev = edge_index.device
    if edge_weight is not None:
        _need_cuda("edge_weight", edge_weight, torch.float32, 1)
    if deg is not None:
        _need_cuda("deg", deg, torch.int64, 1)
        if deg.shape[0] != num_nodes:
            raise ValueError("deg must be [N]")
    norm = torch.empty(E, dtype=torch.float32, device=dev) if out is None else out
    nbytes = _size(lib.pyg_gcn_norm_workspace, E, num_nodes)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    _check(lib.pyg_gcn_norm(_ptr(edge_index), _ptr(edge_weight), E, num_nodes, _ptr(deg), _ptr(norm), _ptr(ws),
                            nbytes, _stream(dev)), "pyg_gcn_norm")
    return norm


def gcn_norm_csr(csr: CSR, out: torch.Tensor | None = None, workspace: torch.Tensor | None = None) -> torch.Tensor:
    """GCN edge norms in CSR slot order (degrees from the CSR rows, weighted by
    csr.weight when present); the result can serve as the weight of a CSR."""
    lib = library()
    dev = csr.rowptr.device
    norm = torch.empty(csr.E, dtype=torch.float32, device=dev) if out is None else out
    nbytes = _size(lib.pyg_gcn_norm_csr_workspace, csr.N)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    c = csr._c()
    _check(lib.pyg_gcn_norm_csr(ctypes.byref(c), _ptr(norm), _ptr(ws), nbytes, _stream(dev)), "pyg_gcn_norm_csr")
    return norm


def gcn_propagate(x: torch.Tensor, csr: CSR, norm_out: torch.Tensor | None = None, out: torch.Tensor | None = None,
                  workspace: torch.Tensor | None = None) -> torch.Tensor:
    """GCN propagate with the normalisation fused in (pyg_gcn_propagate):
    out_i = sum_p norm_p x_col[p], norm_p = d_j^-1/2 w_p d_i^-1/2 formed per slot;
    the norms go to norm_out (CSR slot order) when given."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    if csr.N != N:
        raise ValueError("csr does not match x")
    if norm_out is not None:
        _need_cuda("norm_out", norm_out, torch.float32, 1)
        if norm_out.shape[0] != csr.E:
            raise ValueError("norm_out must be [E]")
    if out is None:
        out = torch.empty_like(x)
    nbytes = _size(lib.pyg_gcn_propagate_workspace, DTYPE[x.dtype], N, F, csr.E, csr.chunk)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, x.device)
    c = csr._c()
    _check(lib.pyg_gcn_propagate(_ptr(x), DTYPE[x.dtype], N, F, ctypes.byref(c), _ptr(norm_out), _ptr(out),
                                 _ptr(workspace), workspace.numel(), _stream(x.device)), "pyg_gcn_propagate")
    return out


def gcn_propagate_workspace_bytes(x: torch.Tensor, csr: CSR) -> int:
    return _size(library().pyg_gcn_propagate_workspace, DTYPE[x.dtype], x.shape[0], x.shape[1], csr.E, csr.chunk)


def gcn_propagate_blocked(x: torch.Tensor, csr: CSR | None, bcsr: CSRBlocks, norm_out: torch.Tensor | None = None,
                          out: torch.Tensor | None = None, workspace: torch.Tensor | None = None) -> torch.Tensor:
    """gcn_propagate over a source-blocked CSR (pyg_gcn_propagate_blocked):
    d from `csr` when given, else from bcsr; the propagate over `bcsr`; the
    norms go to norm_out in bcsr's slot order when given."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    if bcsr.N != N or (csr is not None and (csr.N != N or csr.E != bcsr.E)):
        raise ValueError("csr / bcsr do not match x")
    if norm_out is not None:
        _need_cuda("norm_out", norm_out, torch.float32, 1)
        if norm_out.shape[0] != bcsr.E:
            raise ValueError("norm_out must be [E]")
    if out is None:
        out = torch.empty_like(x)
    nbytes = gcn_propagate_blocked_workspace_bytes(x, bcsr)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, x.device)
    c, b = (csr._c() if csr is not None else None), bcsr._c()
    _check(lib.pyg_gcn_propagate_blocked(_ptr(x), DTYPE[x.dtype], N, F, ctypes.byref(c) if c is not None else None,
                                         ctypes.byref(b),
                                         _ptr(norm_out), _ptr(out), _ptr(workspace), workspace.numel(),
                                         _stream(x.device)), "pyg_gcn_propagate_blocked")
    return out


def gcn_propagate_blocked_workspace_bytes(x: torch.Tensor, bcsr: CSRBlocks) -> int:
    return _size(library().pyg_gcn_propagate_blocked_workspace, DTYPE[x.dtype], x.shape[0], x.shape[1], bcsr.E,
                 bcsr.B, bcsr.chunk)


def propagate_workspace_bytes(x: torch.Tensor, E: int, aggr: str, kernel: str, chunk: int = 0) -> int:
    return _size(library().pyg_propagate_workspace, DTYPE[x.dtype], x.shape[0], x.shape[1], E, AGGR[aggr],
                 KERNEL[kernel], chunk)


def propagate(x: torch.Tensor, edge_index: torch.Tensor | None = None, edge_weight: torch.Tensor | None = None,
              csr: CSR | None = None, aggr: str = "sum", msg: str = "src", kernel: str = "auto",
              out: torch.Tensor | None = None, argmax: torch.Tensor | None = None,
              workspace: torch.Tensor | None = None):
    """Eq. (1) with gamma = identity. Returns (out, argmax or None)."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    dev = x.device
    if edge_index is not None:
        E = _edge_index(edge_index)
    elif csr is not None:
        E = csr.E
    else:
        raise ValueError("need edge_index or csr")
    if csr is not None and (csr.N != N or csr.E != E):
        raise ValueError("csr does not match x / edge_index")
    if edge_weight is not None:
        _need_cuda("edge_weight", edge_weight, torch.float32, 1)
    if aggr not in AGGR or msg not in MSG or kernel not in KERNEL:
        raise ValueError("bad aggr / msg / kernel")
    if out is None:
        out = torch.empty_like(x)
    if aggr == "max" and argmax is None:
        argmax = torch.empty((N, F), dtype=torch.int64, device=dev)
    if aggr != "max":
        argmax = None
    use = "coo" if kernel == "coo" or (kernel == "auto" and csr is None) else "csr"
    chunk = csr.chunk if (csr is not None and use == "csr") else 0
    nbytes = propagate_workspace_bytes(x, E, aggr, use, chunk)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    c = csr._c() if csr is not None else None
    rc = lib.pyg_propagate(_ptr(x), DTYPE[x.dtype], N, F, _ptr(edge_index), E, _ptr(edge_weight),
                           ctypes.byref(c) if c is not None else None, MSG[msg], AGGR[aggr], KERNEL[kernel],
                           _ptr(out), _ptr(argmax), _ptr(workspace), workspace.numel(), _stream(dev))
    _check(rc, "pyg_propagate")
    return out, argmax


def propagate_noalloc(x: torch.Tensor, edge_index: torch.Tensor | None = None,
                      edge_weight: torch.Tensor | None = None, csr: CSR | None = None, aggr: str = "sum",
                      msg: str = "src", kernel: str = "auto", out: torch.Tensor | None = None,
                      argmax: torch.Tensor | None = None):
    """propagate() through pyg_propagate_noalloc: no workspace, the library's
    static per-GPU scratch instead. Allocates nothing when out (and argmax for
    max) are given. Returns (out, argmax or None)."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    E = _edge_index(edge_index) if edge_index is not None else (csr.E if csr is not None else None)
    if E is None:
        raise ValueError("need edge_index or csr")
    if aggr not in AGGR or msg not in MSG or kernel not in KERNEL:
        raise ValueError("bad aggr / msg / kernel")
    if out is None:
        out = torch.empty_like(x)
    if aggr == "max" and argmax is None:
        argmax = torch.empty((N, F), dtype=torch.int64, device=x.device)
    if aggr != "max":
        argmax = None
    c = csr._c() if csr is not None else None
    rc = lib.pyg_propagate_noalloc(_ptr(x), DTYPE[x.dtype], N, F, _ptr(edge_index), E, _ptr(edge_weight),
                                   ctypes.byref(c) if c is not None else None, MSG[msg], AGGR[aggr], KERNEL[kernel],
                                   _ptr(out), _ptr(argmax), _stream(x.device))
    _check(rc, "pyg_propagate_noalloc")
    return out, argmax


def propagate_edge(x: torch.Tensor, edge_attr: torch.Tensor, edge_index: torch.Tensor | None = None,
                   csr: CSR | None = None, msg: str = "edge_add", aggr: str = "sum", kernel: str = "auto",
                   attr_order: str = "coo", out: torch.Tensor | None = None, argmax: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None):
    """Eq. (1) with F-dimensional edge features: phi = x_j + e, max(x_j + e, 0)
    or x_j * e (msg "edge_add", "edge_relu", "edge_mul"). edge_attr [E, F] in
    x's dtype, rows in `attr_order` ("coo": edge id, "csr": CSR slot).
    Returns (out, argmax or None)."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    dev = x.device
    if edge_index is not None:
        E = _edge_index(edge_index)
    elif csr is not None:
        E = csr.E
    else:
        raise ValueError("need edge_index or csr")
    _need_cuda("edge_attr", edge_attr, x.dtype, 2)
    if tuple(edge_attr.shape) != (E, F):
        raise ValueError("edge_attr must be [E, F]")
    if msg not in ("edge_add", "edge_relu", "edge_mul") or aggr not in AGGR or kernel not in KERNEL:
        raise ValueError("bad msg / aggr / kernel")
    out = torch.empty_like(x) if out is None else out
    argmax = (torch.empty((N, F), dtype=torch.int64, device=dev) if argmax is None else argmax) if aggr == "max" else None
    use = "coo" if kernel == "coo" or (kernel == "auto" and csr is None) else "csr"
    nbytes = propagate_workspace_bytes(x, E, aggr, use, csr.chunk if (csr is not None and use == "csr") else 0)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    c = csr._c() if csr is not None else None
    rc = lib.pyg_propagate_edge(_ptr(x), DTYPE[x.dtype], N, F, _ptr(edge_index), E, _ptr(edge_attr), ORDER[attr_order],
                                ctypes.byref(c) if c is not None else None, MSG[msg], AGGR[aggr], KERNEL[kernel],
                                _ptr(out), _ptr(argmax), _ptr(workspace), workspace.numel(), _stream(dev))
    _check(rc, "pyg_propagate_edge")
    return out, argmax


def propagate_edge_encoded(x: torch.Tensor, edge_attr: torch.Tensor, theta_e: torch.Tensor,
                           edge_index: torch.Tensor | None = None, csr: CSR | None = None, msg: str = "edge_add",
                           aggr: str = "sum", kernel: str = "auto", attr_order: str = "coo",
                           out: torch.Tensor | None = None, workspace: torch.Tensor | None = None):
    """propagate_edge with D-dimensional edge features projected to F first:
    e = edge_attr [E, D] @ theta_e [D, F] (the matrix-core transform, e in
    x's dtype), then the edge-feature message with e. Returns (out, argmax
    or None)."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    dev = x.device
    if edge_index is not None:
        E = _edge_index(edge_index)
    elif csr is not None:
        E = csr.E
    else:
        raise ValueError("need edge_index or csr")
    _need_cuda("edge_attr", edge_attr, x.dtype, 2)
    _need_cuda("theta_e", theta_e, x.dtype, 2)
    D = edge_attr.shape[1]
    if edge_attr.shape[0] != E or tuple(theta_e.shape) != (D, F):
        raise ValueError("edge_attr must be [E, D] and theta_e [D, F]")
    if msg not in ("edge_add", "edge_relu", "edge_mul") or aggr not in AGGR or kernel not in KERNEL:
        raise ValueError("bad msg / aggr / kernel")
    out = torch.empty_like(x) if out is None else out
    argmax = torch.empty((N, F), dtype=torch.int64, device=dev) if aggr == "max" else None
    use_csr = kernel == "csr" or (kernel == "auto" and csr is not None)
    nbytes = _size(lib.pyg_propagate_edge_encoded_workspace, DTYPE[x.dtype], N, F, E, D, AGGR[aggr],
                   KERNEL["csr" if use_csr else "coo"], csr.chunk if (csr is not None and use_csr) else 0)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    c = csr._c() if csr is not None else None
    rc = lib.pyg_propagate_edge_encoded(_ptr(x), DTYPE[x.dtype], N, F, _ptr(edge_index), E, _ptr(edge_attr), D,
                                        _ptr(theta_e), ORDER[attr_order], ctypes.byref(c) if c is not None else None,
                                        MSG[msg], AGGR[aggr], KERNEL[kernel], _ptr(out), _ptr(argmax),
                                        _ptr(workspace), workspace.numel(), _stream(dev))
    _check(rc, "pyg_propagate_edge_encoded")
    return out, argmax


def reverse_edges(edge_index: torch.Tensor) -> torch.Tensor:
    """[2,E] edge list with source and target swapped (the transposed graph)."""
    return edge_index.flip(0).contiguous()


def propagate_backward(grad_out: torch.Tensor, x: torch.Tensor | None = None, edge_index: torch.Tensor | None = None,
                       edge_weight: torch.Tensor | None = None, csr: CSR | None = None, csr_t: CSR | None = None,
                       aggr: str = "sum", msg: str = "src", argmax: torch.Tensor | None = None,
                       need_grad_w: bool = False, workspace: torch.Tensor | None = None, w_order: str = "coo"):
    """Gradient of propagate. Returns (grad_x, grad_w or None). csr_t is the
    CSR of reverse_edges(edge_index) built with the same weights (sum/mean).
    grad_w comes in `w_order`: "coo" (edge ids, like edge_weight) or "csr"
    (the slots of csr, like csr.weight)."""
    lib = library()
    _need_cuda("grad_out", grad_out, None, 2)
    if grad_out.dtype not in DTYPE:
        raise ValueError("grad_out must be float32 or bfloat16")
    N, F = grad_out.shape
    dev = grad_out.device
    if edge_index is not None:
        E = _edge_index(edge_index)
    elif csr_t is not None:
        E = csr_t.E
    else:
        raise ValueError("need edge_index or csr_t")
    if x is not None:
        _need_cuda("x", x, grad_out.dtype, 2)
    if edge_weight is not None:
        _need_cuda("edge_weight", edge_weight, torch.float32, 1)
    if w_order not in ORDER:
        raise ValueError("w_order must be 'coo' or 'csr'")
    grad_x = torch.empty_like(grad_out)
    grad_w = torch.empty(E, dtype=torch.float32, device=dev) if need_grad_w else None
    chunk_t = csr_t.chunk if csr_t is not None else 0
    nbytes = _size(lib.pyg_propagate_backward_workspace, DTYPE[grad_out.dtype], N, F, E, AGGR[aggr], chunk_t)
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    c = csr._c() if csr is not None else None
    ct = csr_t._c() if csr_t is not None else None
    rc = lib.pyg_propagate_backward(_ptr(grad_out), _ptr(x), DTYPE[grad_out.dtype], N, F, _ptr(edge_index), E,
                                    _ptr(edge_weight), ctypes.byref(c) if c is not None else None,
                                    ctypes.byref(ct) if ct is not None else None, MSG[msg], AGGR[aggr], _ptr(argmax),
                                    _ptr(grad_x), _ptr(grad_w), ORDER[w_order], _ptr(ws), ws.numel(), _stream(dev))
    _check(rc, "pyg_propagate_backward")
    return grad_x, grad_w


def _edge_values(name, t, E):
    _need_cuda(name, t, torch.float32)
    if t.dim() == 1:
        t = t.view(E, 1) if E else t.view(0, 1)
    if t.dim() != 2 or t.shape[0] != E:
        raise ValueError(f"{name} must be [E, H] or [E]")
    return t


def _softmax_ws(csr: CSR, H: int, workspace):
    nbytes = _size(library().pyg_segment_softmax_workspace, csr.E, csr.N, H, csr.chunk)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, csr.rowptr.device)
    return workspace


def segment_softmax(scores: torch.Tensor, csr: CSR, order: str = "coo", out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None) -> torch.Tensor:
    """Softmax of scores [E, H] (or [E]) over the incoming edges of every
    target, per head; scores and the result are in `order` ("coo": edge id,
    "csr": slot)."""
    lib = library()
    s2 = _edge_values("scores", scores, csr.E)
    H = s2.shape[1]
    out = torch.empty_like(scores) if out is None else out
    ws = _softmax_ws(csr, H, workspace)
    c = csr._c()
    _check(lib.pyg_segment_softmax(_ptr(s2), H, ctypes.byref(c), ORDER[order], _ptr(out), _ptr(ws), ws.numel(),
                                   _stream(csr.rowptr.device)), "pyg_segment_softmax")
    return out


def gat_softmax(a_src: torch.Tensor, a_dst: torch.Tensor, csr: CSR, negative_slope: float = 0.2,
                order: str = "csr", out: torch.Tensor | None = None,
                workspace: torch.Tensor | None = None) -> torch.Tensor:
    """GAT attention coefficients [E, H]: softmax over incoming edges of
    LeakyReLU(a_src[j] + a_dst[i]), scores computed on the fly."""
    lib = library()
    _need_cuda("a_src", a_src, torch.float32, 2)
    _need_cuda("a_dst", a_dst, torch.float32, 2)
    if a_src.shape != a_dst.shape or a_src.shape[0] != csr.N:
        raise ValueError("a_src and a_dst must both be [N, H]")
    H = a_src.shape[1]
    out = torch.empty((csr.E, H), dtype=torch.float32, device=a_src.device) if out is None else out
    ws = _softmax_ws(csr, H, workspace)
    c = csr._c()
    _check(lib.pyg_gat_softmax(_ptr(a_src), _ptr(a_dst), H, ctypes.c_float(negative_slope), ctypes.byref(c),
                               ORDER[order], _ptr(out), _ptr(ws), ws.numel(), _stream(a_src.device)),
           "pyg_gat_softmax")
    return out


def segment_softmax_backward(alpha: torch.Tensor, grad_alpha: torch.Tensor, csr: CSR, order: str = "coo",
                             out: torch.Tensor | None = None, workspace: torch.Tensor | None = None) -> torch.Tensor:
    """Gradient of segment_softmax w.r.t. its scores."""
    lib = library()
    a2 = _edge_values("alpha", alpha, csr.E)
    g2 = _edge_values("grad_alpha", grad_alpha, csr.E)
    if g2.shape != a2.shape:
        raise ValueError("grad_alpha must match alpha")
    H = a2.shape[1]
    out = torch.empty_like(alpha) if out is None else out
    ws = _softmax_ws(csr, H, workspace)
    c = csr._c()
    _check(lib.pyg_segment_softmax_backward(_ptr(a2), _ptr(g2), H, ctypes.byref(c), ORDER[order], _ptr(out),
                                            _ptr(ws), ws.numel(), _stream(csr.rowptr.device)),
           "pyg_segment_softmax_backward")
    return out


def propagate_heads(x: torch.Tensor, csr: CSR, alpha: torch.Tensor, heads: int, out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None) -> torch.Tensor:
    """out[i, h*C:(h+1)*C] = sum over CSR slots p of row i of alpha[p, h] * x[col[p], h*C:(h+1)*C];
    alpha [E, H] in CSR slot order."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE:
        raise ValueError("x must be float32 or bfloat16")
    N, F = x.shape
    if heads <= 0 or F % heads:
        raise ValueError("the feature width must be a multiple of heads")
    if csr.N != N:
        raise ValueError("csr does not match x")
    a2 = _edge_values("alpha", alpha, csr.E)
    if a2.shape[1] != heads:
        raise ValueError("alpha must be [E, heads]")
    C = F // heads
    out = torch.empty_like(x) if out is None else out
    nbytes = _size(lib.pyg_propagate_heads_workspace, DTYPE[x.dtype], N, heads, C, csr.E, csr.chunk)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, x.device)
    c = csr._c()
    _check(lib.pyg_propagate_heads(_ptr(x), DTYPE[x.dtype], N, heads, C, ctypes.byref(c), _ptr(a2), _ptr(out),
                                   _ptr(workspace), workspace.numel(), _stream(x.device)), "pyg_propagate_heads")
    return out


def propagate_edge_backward(grad_out: torch.Tensor, x: torch.Tensor | None, edge_attr: torch.Tensor | None, csr: CSR,
                            msg: str, aggr: str = "sum", order: str = "csr", csr_t: CSR | None = None,
                            map_t: torch.Tensor | None = None, edge_index: torch.Tensor | None = None,
                            argmax: torch.Tensor | None = None, need_grad_x: bool = True,
                            need_grad_edge: bool = True, workspace: torch.Tensor | None = None):
    """Gradients of propagate_edge (fp32 or bf16, the dtype of grad_out):
    (grad_x [N, F] or None, grad_edge_attr [E, F] in `order` or None). Sum /
    mean need csr_t for grad_x (map_t optional); max needs edge_index and the
    forward's argmax."""
    lib = library()
    _need_cuda("grad_out", grad_out, None, 2)
    if grad_out.dtype not in DTYPE:
        raise ValueError("grad_out must be float32 or bfloat16")
    dt = grad_out.dtype
    N, F = grad_out.shape
    E = csr.E
    if msg not in ("edge_add", "edge_relu", "edge_mul") or aggr not in AGGR or order not in ORDER:
        raise ValueError("bad msg / aggr / order")
    if msg != "edge_add":
        _need_cuda("x", x, dt, 2)
        _need_cuda("edge_attr", edge_attr, dt, 2)
        if tuple(edge_attr.shape) != (E, F):
            raise ValueError("edge_attr must be [E, F]")
    if aggr == "max":
        _need_cuda("argmax", argmax, torch.int64, 2)
        if edge_index is None:
            raise ValueError("max needs edge_index")
        _edge_index(edge_index)
    elif need_grad_x and csr_t is None:
        raise ValueError("sum / mean need csr_t for grad_x")
    dev = grad_out.device
    gx = torch.empty_like(grad_out) if need_grad_x else None
    ge = torch.empty((E, F), dtype=dt, device=dev) if need_grad_edge else None
    chunk_t = csr_t.chunk if (csr_t is not None and aggr != "max" and need_grad_x) else 0
    nbytes = _size(lib.pyg_propagate_edge_backward_workspace, DTYPE[dt], N, F, E, MSG[msg], AGGR[aggr], chunk_t)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    c = csr._c()
    ct = csr_t._c() if csr_t is not None else None
    _check(lib.pyg_propagate_edge_backward(_ptr(grad_out), _ptr(x), _ptr(edge_attr), DTYPE[dt], N, F,
                                           _ptr(edge_index), ctypes.byref(c), ctypes.byref(ct) if ct else None,
                                           _ptr(_map_t(map_t, E)), ORDER[order], MSG[msg], AGGR[aggr], _ptr(argmax),
                                           _ptr(gx), _ptr(ge), _ptr(workspace), workspace.numel(), _stream(dev)),
           "pyg_propagate_edge_backward")
    return gx, ge


def csr_transpose_map(csr: CSR, csr_t: CSR, out: torch.Tensor | None = None,
                      workspace: torch.Tensor | None = None) -> torch.Tensor:
    """int32 [E]: for each slot of csr_t (the CSR of the reversed edges) the
    slot of csr holding the same edge. Made once per graph, passed as map_t
    to the attention backward."""
    lib = library()
    if csr.N != csr_t.N or csr.E != csr_t.E:
        raise ValueError("csr and csr_t must describe the same graph")
    dev = csr.rowptr.device
    if out is None:
        out = torch.empty(csr.E, dtype=torch.int32, device=dev)
    else:
        _need_cuda("out", out, torch.int32, 1)
        if out.shape[0] != csr.E:
            raise ValueError("out must be [E]")
    nbytes = _size(lib.pyg_csr_transpose_map_workspace, csr.E)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    c, ct = csr._c(), csr_t._c()
    _check(lib.pyg_csr_transpose_map(ctypes.byref(c), ctypes.byref(ct), _ptr(out), _ptr(workspace), workspace.numel(),
                                     _stream(dev)), "pyg_csr_transpose_map")
    return out


def _map_t(map_t, E):
    if map_t is None:
        return None
    _need_cuda("map_t", map_t, torch.int32, 1)
    if map_t.shape[0] != E:
        raise ValueError("map_t must be [E]")
    return map_t


def propagate_heads_backward(grad_out: torch.Tensor, x: torch.Tensor | None, csr: CSR, csr_t: CSR,
                             alpha: torch.Tensor, heads: int, need_grad_x: bool = True, need_grad_alpha: bool = True,
                             workspace: torch.Tensor | None = None, out: tuple | None = None,
                             map_t: torch.Tensor | None = None):
    """Gradients of propagate_heads: (grad_x [N, H*C] in grad_out's dtype or
    None, grad_alpha fp32 [E, H] in CSR slot order or None). `out` may bring
    both result tensors (grad_x, grad_alpha) preallocated; `map_t` is
    csr_transpose_map(csr, csr_t), else made on every call."""
    lib = library()
    _need_cuda("grad_out", grad_out, None, 2)
    if grad_out.dtype not in DTYPE:
        raise ValueError("grad_out must be float32 or bfloat16")
    N, F = grad_out.shape
    if heads <= 0 or F % heads:
        raise ValueError("the feature width must be a multiple of heads")
    C = F // heads
    a2 = _edge_values("alpha", alpha, csr.E)
    if need_grad_alpha:
        _need_cuda("x", x, grad_out.dtype, 2)
    dev = grad_out.device
    if out is not None:
        gx, ga = out
        if need_grad_x:
            _need_cuda("out[0]", gx, grad_out.dtype, 2)
            if tuple(gx.shape) != (N, F):
                raise ValueError("out[0] must match grad_out's shape")
        if need_grad_alpha:
            _need_cuda("out[1]", ga, torch.float32, 2)
            if tuple(ga.shape) != (csr.E, heads):
                raise ValueError("out[1] must be [E, heads]")
    else:
        gx = torch.empty_like(grad_out) if need_grad_x else None
        ga = torch.empty((csr.E, heads), dtype=torch.float32, device=dev) if need_grad_alpha else None
    nbytes = _size(lib.pyg_propagate_heads_backward_workspace, DTYPE[grad_out.dtype], N, heads, C, csr.E, csr_t.chunk)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, dev)
    c, ct = csr._c(), csr_t._c()
    mt = _map_t(map_t, csr.E)
    _check(lib.pyg_propagate_heads_backward(_ptr(grad_out), _ptr(x if need_grad_alpha else None), DTYPE[grad_out.dtype],
                                            N, heads, C, ctypes.byref(c), ctypes.byref(ct), _ptr(mt), _ptr(a2), _ptr(gx),
                                            _ptr(ga), _ptr(workspace), workspace.numel(), _stream(dev)),
           "pyg_propagate_heads_backward")
    return gx, ga


def gat_scores_backward(a_src: torch.Tensor, a_dst: torch.Tensor, csr: CSR, csr_t: CSR, grad_scores: torch.Tensor,
                        negative_slope: float = 0.2, workspace: torch.Tensor | None = None,
                        out: tuple | None = None, map_t: torch.Tensor | None = None):
    """Gradients of GAT's edge scores w.r.t. the node logits: (grad_a_src,
    grad_a_dst), fp32 [N, H]; grad_scores [E, H] in CSR slot order. `out`
    may bring both result tensors preallocated; `map_t` as for
    propagate_heads_backward."""
    lib = library()
    _need_cuda("a_src", a_src, torch.float32, 2)
    _need_cuda("a_dst", a_dst, torch.float32, 2)
    N, H = a_src.shape
    g2 = _edge_values("grad_scores", grad_scores, csr.E)
    if out is not None:
        gs, gd = out
        for name, t in (("out[0]", gs), ("out[1]", gd)):
            _need_cuda(name, t, torch.float32, 2)
            if t.shape != a_src.shape:
                raise ValueError(f"{name} must be [N, heads]")
    else:
        gs, gd = torch.empty_like(a_src), torch.empty_like(a_dst)
    nbytes = _size(lib.pyg_gat_scores_backward_workspace, N, H, csr.E, csr_t.chunk)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, a_src.device)
    c, ct = csr._c(), csr_t._c()
    mt = _map_t(map_t, csr.E)
    _check(lib.pyg_gat_scores_backward(_ptr(a_src), _ptr(a_dst), H, ctypes.c_float(negative_slope), ctypes.byref(c),
                                       ctypes.byref(ct), _ptr(mt), _ptr(g2), _ptr(gs), _ptr(gd), _ptr(workspace),
                                       workspace.numel(), _stream(a_src.device)), "pyg_gat_scores_backward")
    return gs, gd


def dense_transform(x: torch.Tensor, theta: torch.Tensor, out_dtype=torch.float32, out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None) -> torch.Tensor:
    """x [N, Fi] times theta [Fi, Fo] (both bf16 or both float32) on the
    matrix cores, fp32 accumulation; the result in out_dtype (float32 or
    bfloat16)."""
    lib = library()
    _need_cuda("x", x, None, 2)
    if x.dtype not in DTYPE or out_dtype not in DTYPE:
        raise ValueError("x and out must be float32 or bfloat16")
    _need_cuda("theta", theta, x.dtype, 2)
    N, Fi = x.shape
    if theta.shape[0] != Fi:
        raise ValueError("theta must be [Fi, Fo]")
    Fo = theta.shape[1]
    out = torch.empty((N, Fo), dtype=out_dtype, device=x.device) if out is None else out
    nbytes = _size(lib.pyg_dense_transform_workspace, Fi, Fo)
    if workspace is None or workspace.numel() < nbytes:
        workspace = _workspace(nbytes, x.device)
    _check(lib.pyg_dense_transform(_ptr(x), DTYPE[x.dtype], N, Fi, _ptr(theta), Fo, _ptr(out), DTYPE[out.dtype],
                                   _ptr(workspace), workspace.numel(), _stream(x.device)), "pyg_dense_transform")
    return out


def global_pool(x: torch.Tensor, batch: torch.Tensor, num_graphs: int, aggr: str = "sum",
                out: torch.Tensor | None = None, argmax: torch.Tensor | None = None,
                workspace: torch.Tensor | None = None):
    """Per-graph readout over a sorted assignment vector. Returns (out, argmax or None)."""
    lib = library()
    _need_cuda("x", x, None, 2)
    _need_cuda("batch", batch, torch.int64, 1)
    N, F = x.shape
    if batch.shape[0] != N:
        raise ValueError("batch must be [N]")
    dev = x.device
    if out is None:
        out = torch.empty((num_graphs, F), dtype=x.dtype, device=dev)
    if aggr == "max" and argmax is None:
        argmax = torch.empty((num_graphs, F), dtype=torch.int64, device=dev)
    if aggr != "max":
        argmax = None
    nbytes = _size(lib.pyg_global_pool_workspace, DTYPE[x.dtype], N, F, num_graphs, AGGR[aggr])
    ws = workspace if workspace is not None and workspace.numel() >= nbytes else _workspace(nbytes, dev)
    _check(lib.pyg_global_pool(_ptr(x), DTYPE[x.dtype], N, F, _ptr(batch), num_graphs, AGGR[aggr], _ptr(out),
                               _ptr(argmax), _ptr(ws), nbytes, _stream(dev)), "pyg_global_pool")
    return out, argmax


def validate_coo(edge_index: torch.Tensor, num_nodes: int) -> int:
    """Number of edge_index entries outside [0, num_nodes) (synchronises)."""
    E = _edge_index(edge_index)
    bad = torch.empty(1, dtype=torch.int64, device=edge_index.device)
    _check(library().pyg_validate_coo(_ptr(edge_index), E, num_nodes, _ptr(bad), _stream(edge_index.device)),
           "pyg_validate_coo")
    return int(bad.item())


def validate_batch(batch: torch.Tensor, num_graphs: int) -> int:
    """Number of batch entries out of range or out of order (synchronises)."""
    _need_cuda("batch", batch, torch.int64, 1)
    bad = torch.empty(1, dtype=torch.int64, device=batch.device)
    _check(library().pyg_validate_batch(_ptr(batch), batch.shape[0], num_graphs, _ptr(bad), _stream(batch.device)),
           "pyg_validate_batch")
    return int(bad.item())


class Graph:
    """A graph prepared once for repeated propagates with gradients: the
    forward CSR and the CSR of the transposed graph (both with the weights)."""

    def __init__(self, edge_index: torch.Tensor, num_nodes: int, edge_weight: torch.Tensor | None = None):
        self.edge_index = edge_index
        self.N = num_nodes
        self.edge_weight = edge_weight
        self.csr = coo_to_csr(edge_index, num_nodes, edge_weight)
        self.csr_t = coo_to_csr(reverse_edges(edge_index), num_nodes, edge_weight)
        self._map_t = None

    @property
    def plain(self) -> CSR:
        """The forward CSR without weights (attention and edge messages)."""
        c = self.csr
        return CSR(c.rowptr, c.col, c.perm, None, c.N, c.E, c.chunk)

    @property
    def plain_t(self) -> CSR:
        """The CSR of the transposed graph without weights."""
        c = self.csr_t
        return CSR(c.rowptr, c.col, c.perm, None, c.N, c.E, c.chunk)

    @property
    def map_t(self) -> torch.Tensor:
        """Transpose map of (csr, csr_t), made on first use."""
        if self._map_t is None:
            self._map_t = csr_transpose_map(self.csr, self.csr_t)
        return self._map_t


class Propagate(torch.autograd.Function):
    """Differentiable propagate on the CSR segment kernel; the backward runs
    pyg_propagate_backward (gradients for x and, when weighted, the weights).
    Use as Propagate.apply(x, edge_weight_or_None, graph, aggr, msg)."""

    @staticmethod
    def forward(ctx, x, edge_weight, graph: Graph, aggr: str = "sum", msg: str = "src"):
        # without a weight the message is x_j (or x_j - x_i), whatever weights the Graph was built with
        csr = graph.plain
        if edge_weight is not None:
            # the CSR carries the weights in slot order: refresh them from the current tensor
            csr = CSR(csr.rowptr, csr.col, csr.perm, gather_edges(csr.perm, edge_weight.detach().contiguous()),
                      csr.N, csr.E, csr.chunk)
        out, argmax = propagate(x.detach().contiguous(), graph.edge_index, None if edge_weight is None else
                                edge_weight.detach(), csr=csr, aggr=aggr, msg=msg)
        ctx.graph, ctx.aggr, ctx.msg = graph, aggr, msg
        ctx.save_for_backward(x, edge_weight, argmax)
        return out

    @staticmethod
    def backward(ctx, grad_out):
        x, edge_weight, argmax = ctx.saved_tensors
        g = ctx.graph
        csr, csr_t = g.plain, g.plain_t
        if edge_weight is not None:
            w = edge_weight.detach().contiguous()
            csr = CSR(csr.rowptr, csr.col, csr.perm, gather_edges(csr.perm, w), csr.N, csr.E, csr.chunk)
            csr_t = CSR(csr_t.rowptr, csr_t.col, csr_t.perm, gather_edges(csr_t.perm, w), csr_t.N, csr_t.E,
                        csr_t.chunk)
        need_w = edge_weight is not None and ctx.needs_input_grad[1]
        gx, gw = propagate_backward(grad_out.contiguous(), x.detach().contiguous(), g.edge_index,
                                    None if edge_weight is None else edge_weight.detach(), csr, csr_t,
                                    ctx.aggr, ctx.msg, argmax, need_grad_w=need_w)
        return gx, gw, None, None, None


class GATAttention(torch.autograd.Function):
    """GAT's attention aggregation (Section 2): coefficients alpha =
    softmax over each target's incoming edges of LeakyReLU(a_src[j] +
    a_dst[i]) per head, then out_i = sum_j alpha_{j,i} x_j per head block.
    Forward: gat_softmax + propagate_heads; backward: propagate_heads_backward,
    segment_softmax_backward, gat_scores_backward (all in CSR slot order).
    Use as GATAttention.apply(x [N, H*C], a_src [N, H], a_dst [N, H], graph,
    negative_slope); fp32 or bf16 x, fp32 logits."""

    @staticmethod
    def forward(ctx, x, a_src, a_dst, graph: Graph, negative_slope: float = 0.2):
        H = a_src.shape[1]
        csr = graph.plain
        alpha = gat_softmax(a_src.detach().contiguous(), a_dst.detach().contiguous(), csr, negative_slope, "csr")
        out = propagate_heads(x.detach().contiguous(), csr, alpha, H)
        ctx.graph, ctx.slope = graph, negative_slope
        ctx.save_for_backward(x, a_src, a_dst, alpha)
        return out

    @staticmethod
    def backward(ctx, grad_out):
        x, a_src, a_dst, alpha = ctx.saved_tensors
        g = ctx.graph
        H = a_src.shape[1]
        need_logits = ctx.needs_input_grad[1] or ctx.needs_input_grad[2]
        gx, galpha = propagate_heads_backward(grad_out.contiguous().to(x.dtype), x.detach().contiguous(), g.plain,
                                              g.csr_t, alpha, H, need_grad_x=ctx.needs_input_grad[0],
                                              need_grad_alpha=need_logits, map_t=g.map_t)
        ga_s = ga_d = None
        if need_logits:
            gscore = segment_softmax_backward(alpha, galpha, g.plain, "csr")
            ga_s, ga_d = gat_scores_backward(a_src.detach().contiguous(), a_dst.detach().contiguous(), g.plain,
                                             g.csr_t, gscore, ctx.slope, map_t=g.map_t)
        return gx, ga_s, ga_d, None, None


class PropagateEdge(torch.autograd.Function):
    """Differentiable propagate with F-dimensional edge features (Eq. (1)):
    phi = x_j + e, max(x_j + e, 0) or x_j * e on the CSR segment kernel;
    gradients for x and the edge features (COO edge order) by
    pyg_propagate_edge_backward (fp32 or bf16). Use as
    PropagateEdge.apply(x, edge_attr, graph, msg, aggr)."""

    @staticmethod
    def forward(ctx, x, edge_attr, graph: Graph, msg: str = "edge_add", aggr: str = "sum"):
        out, argmax = propagate_edge(x.detach().contiguous(), edge_attr.detach().contiguous(), graph.edge_index,
                                     graph.plain, msg, aggr, "csr", "coo")
        ctx.graph, ctx.msg, ctx.aggr = graph, msg, aggr
        ctx.save_for_backward(x, edge_attr, argmax)
        return out

    @staticmethod
    def backward(ctx, grad_out):
        x, edge_attr, argmax = ctx.saved_tensors
        g = ctx.graph
        gx, ge = propagate_edge_backward(grad_out.contiguous(), x.detach().contiguous(),
                                         edge_attr.detach().contiguous(), g.plain, ctx.msg, ctx.aggr, "coo",
                                         csr_t=g.csr_t, edge_index=g.edge_index, argmax=argmax,
                                         need_grad_x=ctx.needs_input_grad[0],
                                         need_grad_edge=ctx.needs_input_grad[1])
        return gx, ge, None, None, None
