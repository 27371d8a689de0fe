"""MI355X (gfx950) propagate path of PyTorch Geometric, as a C-ABI HIP library.

This package is a thin Python binding over ``libpyg_mi355x.so``: it checks
tensor arguments, marshals pointers through ctypes and passes torch's current
HIP stream. Every step of the computation runs in the library's own HIP
kernels; PyTorch only provides device memory and streams. There is no CPU
fallback: without the built library every call raises.

The C entry points and their semantics are documented in
``include/pyg_mi355x.h``; the names here mirror them without the ``pyg_``
prefix.
"""
from __future__ import annotations

from .binding import (  # noqa: F401
    CSR,
    CSRBlocks,
    GATAttention,
    Graph,
    Propagate,
    PropagateEdge,
    LibraryMissing,
    PygError,
    abi_version,
    coo_to_csr,
    coo_to_csr_blocked,
    coo_to_csr_blocked_workspace_bytes,
    csr_blocks,
    csr_transpose_map,
    degree,
    degree_csr,
    degree_csr_blocks,
    dense_transform,
    gat_scores_backward,
    gat_softmax,
    gather_edges,
    gcn_norm,
    gcn_norm_csr,
    gcn_propagate,
    gcn_propagate_blocked,
    gcn_propagate_blocked_workspace_bytes,
    gcn_propagate_workspace_bytes,
    global_pool,
    library,
    library_path,
    propagate,
    propagate_backward,
    propagate_blocked,
    propagate_blocked_workspace_bytes,
    propagate_edge,
    propagate_edge_backward,
    propagate_edge_encoded,
    propagate_heads,
    propagate_heads_backward,
    propagate_noalloc,
    propagate_workspace_bytes,
    reverse_edges,
    segment_softmax,
    segment_softmax_backward,
    strerror,
    validate_batch,
    validate_coo,
)
