// C ABI entry points for propagate and global pooling: host-side argument
// checks, workspace sizing and kernel choice. Every check runs before any
// device work is enqueued.
#include "common.hpp"

namespace pyg {
namespace {

constexpr int64_t kMax32 = int64_t(1) << 31;

bool valid_dtype(int dt) { return dt == PYG_F32 || dt == PYG_BF16; }
bool valid_aggr(int a) { return a == PYG_SUM || a == PYG_MEAN || a == PYG_MAX; }
int64_t dtype_size(int dt) { return dt == PYG_BF16 ? 2 : 4; }

bool overlaps(const void *a, int64_t abytes, const void *b, int64_t bbytes) {
    if (!a || !b || abytes <= 0 || bbytes <= 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + static_cast<uintptr_t>(bbytes) && b0 < a0 + static_cast<uintptr_t>(abytes);
}

// Graph offsets of a sorted assignment vector: ptr[g] = first n with batch[n] >= g.
__global__ void k_batch_ptr(const int64_t *__restrict__ batch, int64_t N, int64_t B, int64_t *__restrict__ ptr) {
    for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g <= B; g += (int64_t)gridDim.x * blockDim.x) {
        int64_t lo = 0, hi = N;
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo) / 2;
            if (batch[mid] < g) lo = mid + 1;
            else hi = mid;
        }
        ptr[g] = lo;
    }
}

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" const char *pyg_strerror(int status) {
    switch (status) {
        case PYG_OK: return "success";
        case PYG_ERR_INVALID_ARG: return "invalid argument";
        case PYG_ERR_INDEX_RANGE: return "index out of range";
        case PYG_ERR_WORKSPACE: return "workspace too small";
        case PYG_ERR_HIP: return "HIP runtime or launch error";
        case PYG_ERR_UNSUPPORTED: return "unsupported size or combination";
        default: return "unknown status";
    }
}

extern "C" int pyg_abi_version(void) { return 2; }

extern "C" int pyg_propagate_workspace(int dtype, int64_t N, int64_t F, int64_t E, int aggr, int kernel, int64_t chunk,
                                       size_t *bytes) {
    if (!bytes || !valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || E < 0 || chunk < 0) return PYG_ERR_INVALID_ARG;
    if (kernel != PYG_KERNEL_AUTO && kernel != PYG_KERNEL_COO_ATOMIC && kernel != PYG_KERNEL_CSR_SEGMENT)
        return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || E >= kMax32) return PYG_ERR_UNSUPPORTED;
    const size_t coo = coo_workspace(dtype, N, F, aggr);
    const size_t csr = segment_workspace(E, F, aggr, chunk, N);
    *bytes = kernel == PYG_KERNEL_COO_ATOMIC ? coo : (kernel == PYG_KERNEL_CSR_SEGMENT ? csr : (coo > csr ? coo : csr));
    return PYG_OK;
}

namespace pyg {
int propagate_check(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                    const float *edge_weight, const pyg_csr *csr, int msg, int aggr, int kernel, const void *out,
                    const int64_t *argmax, size_t *need) {
    if (!valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || E < 0) return PYG_ERR_INVALID_ARG;
    if (msg != PYG_MSG_SRC && msg != PYG_MSG_DIFF) return PYG_ERR_INVALID_ARG;
    if (kernel != PYG_KERNEL_AUTO && kernel != PYG_KERNEL_COO_ATOMIC && kernel != PYG_KERNEL_CSR_SEGMENT)
        return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || E >= kMax32) return PYG_ERR_UNSUPPORTED;
    if (msg == PYG_MSG_DIFF && edge_weight) return PYG_ERR_INVALID_ARG;
    if ((aggr == PYG_MAX) != (argmax != nullptr) && N * F > 0) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_MAX && argmax) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && (!x || !out)) return PYG_ERR_INVALID_ARG;
    if (E > 0 && N == 0) return PYG_ERR_INVALID_ARG;
    const int64_t xbytes = N * F * dtype_size(dtype);
    if (overlaps(x, xbytes, out, xbytes)) return PYG_ERR_INVALID_ARG;
    if (argmax && (overlaps(argmax, N * F * 8, x, xbytes) || overlaps(argmax, N * F * 8, out, xbytes)))
        return PYG_ERR_INVALID_ARG;
    if (kernel == PYG_KERNEL_CSR_SEGMENT && !csr) return PYG_ERR_INVALID_ARG;
    const bool use_csr = kernel == PYG_KERNEL_CSR_SEGMENT || (kernel == PYG_KERNEL_AUTO && csr);
    if (use_csr) {
        if (csr->N != N || csr->E != E || !csr->rowptr || csr->chunk < 0) return PYG_ERR_INVALID_ARG;
        if (E > 0 && (!csr->col || (aggr == PYG_MAX && !csr->perm))) return PYG_ERR_INVALID_ARG;
        if (edge_weight && !csr->weight) return PYG_ERR_INVALID_ARG;
        if (msg == PYG_MSG_DIFF && csr->weight) return PYG_ERR_INVALID_ARG;
    } else if (E > 0 && !edge_index) {
        return PYG_ERR_INVALID_ARG;
    }
    return pyg_propagate_workspace(dtype, N, F, E, aggr, use_csr ? PYG_KERNEL_CSR_SEGMENT : PYG_KERNEL_COO_ATOMIC,
                                   use_csr ? csr->chunk : 0, need);
}
}  // namespace pyg

extern "C" int pyg_propagate(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                             const float *edge_weight, const pyg_csr *csr, int msg, int aggr, int kernel, void *out,
                             int64_t *argmax, void *ws, size_t ws_bytes, void *stream) {
    size_t need = 0;
    PYG_TRY(propagate_check(x, dtype, N, F, edge_index, E, edge_weight, csr, msg, aggr, kernel, out, argmax, &need));
    if (ws_bytes < need || (need > 256 && !ws)) return PYG_ERR_WORKSPACE;
    if (N * F == 0) return PYG_OK;
    const bool use_csr = kernel == PYG_KERNEL_CSR_SEGMENT || (kernel == PYG_KERNEL_AUTO && csr);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (!use_csr) return coo_propagate(x, dtype, N, F, edge_index, E, edge_weight, msg, aggr, out, argmax, ws, ws_bytes, s);
    SegmentArgs a{};
    a.x = x;
    a.dtype = dtype;
    a.F = F;
    a.rowptr = csr->rowptr;
    a.col = csr->col;
    a.weight = csr->weight;
    a.perm = csr->perm;
    a.n_rows = N;
    a.E = E;
    a.msg = msg;
    a.aggr = aggr;
    a.chunk = csr->chunk;
    a.sentinel = E;
    a.out = out;
    a.argmax = argmax;
    a.hint = true;
    return segment_reduce(a, ws, ws_bytes, s);
}

extern "C" int pyg_propagate_blocked_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t B, int aggr,
                                               int64_t chunk, size_t *bytes) {
    if (!bytes || !valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || E < 0 || chunk < 0)
        return PYG_ERR_INVALID_ARG;
    if (B < 2 || B > 32) return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || E >= kMax32) return PYG_ERR_UNSUPPORTED;
    *bytes = segment_blocked_workspace(E, N, F, B, aggr, chunk);
    return PYG_OK;
}

extern "C" int pyg_propagate_blocked(const void *x, int dtype, int64_t N, int64_t F, const pyg_csr_blocks *bcsr,
                                     int msg, int aggr, void *out, int64_t *argmax, void *ws, size_t ws_bytes,
                                     void *stream) {
    if (!valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || !bcsr) return PYG_ERR_INVALID_ARG;
    if (msg != PYG_MSG_SRC && msg != PYG_MSG_DIFF) return PYG_ERR_INVALID_ARG;
    const int64_t E = bcsr->E, B = bcsr->B;
    if (bcsr->N != N || E < 0 || !bcsr->rowptr || bcsr->chunk < 0) return PYG_ERR_INVALID_ARG;
    if (B < 2 || B > 32) return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || E >= kMax32) return PYG_ERR_UNSUPPORTED;
    if ((aggr == PYG_MAX) != (argmax != nullptr) && N * F > 0) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_MAX && argmax) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && (!x || !out)) return PYG_ERR_INVALID_ARG;
    if (E > 0 && (N == 0 || !bcsr->col || (aggr == PYG_MAX && !bcsr->perm))) return PYG_ERR_INVALID_ARG;
    if (msg == PYG_MSG_DIFF && bcsr->weight) return PYG_ERR_INVALID_ARG;
    const int64_t xbytes = N * F * dtype_size(dtype);
    if (overlaps(x, xbytes, out, xbytes)) return PYG_ERR_INVALID_ARG;
    if (argmax && (overlaps(argmax, N * F * 8, x, xbytes) || overlaps(argmax, N * F * 8, out, xbytes)))
        return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && ((F * dtype_size(dtype)) % 16 != 0 || reinterpret_cast<uintptr_t>(x) % 16 != 0 ||
                      reinterpret_cast<uintptr_t>(out) % 16 != 0))
        return PYG_ERR_UNSUPPORTED;
    size_t need = 0;
    PYG_TRY(pyg_propagate_blocked_workspace(dtype, N, F, E, B, aggr, bcsr->chunk, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    if (N * F == 0) return PYG_OK;
    SegmentArgs a{};
    a.x = x;
    a.dtype = dtype;
    a.F = F;
    a.rowptr = bcsr->rowptr;
    a.col = bcsr->col;
    a.weight = bcsr->weight;
    a.perm = bcsr->perm;
    a.n_rows = N;
    a.E = E;
    a.msg = msg;
    a.aggr = aggr;
    a.chunk = bcsr->chunk;
    a.sentinel = E;
    a.out = out;
    a.argmax = argmax;
    return segment_reduce_blocked(a, B, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

namespace {
// Argument checks of the edge-feature propagate, shared with the encoded
// variant (which must reject its arguments before any device work):
// edge_attr and attr_bytes are the features the caller passes.
int check_edge_args(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                    const void *edge_attr, int64_t attr_bytes, int attr_order, const pyg_csr *csr, int msg, int aggr,
                    int kernel, const void *out, const int64_t *argmax, bool *use_csr) {
    if (!valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || E < 0) return PYG_ERR_INVALID_ARG;
    if (msg != PYG_MSG_EDGE_ADD && msg != PYG_MSG_EDGE_RELU && msg != PYG_MSG_EDGE_MUL) return PYG_ERR_INVALID_ARG;
    if (attr_order != PYG_ORDER_COO && attr_order != PYG_ORDER_CSR) return PYG_ERR_INVALID_ARG;
    if (kernel != PYG_KERNEL_AUTO && kernel != PYG_KERNEL_COO_ATOMIC && kernel != PYG_KERNEL_CSR_SEGMENT)
        return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || E >= kMax32) return PYG_ERR_UNSUPPORTED;
    if ((aggr == PYG_MAX) != (argmax != nullptr) && N * F > 0) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_MAX && argmax) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && (!x || !out)) return PYG_ERR_INVALID_ARG;
    if (attr_bytes > 0 && !edge_attr) return PYG_ERR_INVALID_ARG;
    if (E > 0 && N == 0) return PYG_ERR_INVALID_ARG;
    const int64_t xbytes = N * F * dtype_size(dtype);
    if (overlaps(x, xbytes, out, xbytes) || overlaps(edge_attr, attr_bytes, out, xbytes)) return PYG_ERR_INVALID_ARG;
    if (argmax && (overlaps(argmax, N * F * 8, x, xbytes) || overlaps(argmax, N * F * 8, out, xbytes)))
        return PYG_ERR_INVALID_ARG;
    if (kernel == PYG_KERNEL_CSR_SEGMENT && !csr) return PYG_ERR_INVALID_ARG;
    *use_csr = kernel == PYG_KERNEL_CSR_SEGMENT || (kernel == PYG_KERNEL_AUTO && csr);
    if (*use_csr) {
        if (csr->N != N || csr->E != E || !csr->rowptr || csr->chunk < 0) return PYG_ERR_INVALID_ARG;
        if (E > 0 && (!csr->col || ((aggr == PYG_MAX || attr_order == PYG_ORDER_COO) && !csr->perm)))
            return PYG_ERR_INVALID_ARG;
    } else {
        if (E > 0 && !edge_index) return PYG_ERR_INVALID_ARG;
        if (attr_order != PYG_ORDER_COO) return PYG_ERR_INVALID_ARG;  // the COO kernel reads edges in COO order
    }
    return PYG_OK;
}
}  // namespace

extern "C" int pyg_propagate_edge(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                                  const void *edge_attr, int attr_order, const pyg_csr *csr, int msg, int aggr,
                                  int kernel, void *out, int64_t *argmax, void *ws, size_t ws_bytes, void *stream) {
    bool use_csr = false;
    PYG_TRY(check_edge_args(x, dtype, N, F, edge_index, E, edge_attr, E * F * dtype_size(dtype), attr_order, csr,
                            msg, aggr, kernel, out, argmax, &use_csr));
    size_t need;
    PYG_TRY(pyg_propagate_workspace(dtype, N, F, E, aggr, use_csr ? PYG_KERNEL_CSR_SEGMENT : PYG_KERNEL_COO_ATOMIC,
                                    use_csr ? csr->chunk : 0, &need));
    if (ws_bytes < need || (need > 256 && !ws)) return PYG_ERR_WORKSPACE;
    if (N * F == 0) return PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (!use_csr)
        return coo_propagate(x, dtype, N, F, edge_index, E, nullptr, msg, aggr, out, argmax, ws, ws_bytes, s, edge_attr);
    SegmentArgs a{};
    a.x = x;
    a.dtype = dtype;
    a.F = F;
    a.rowptr = csr->rowptr;
    a.col = csr->col;
    a.perm = csr->perm;
    a.edge_attr = E > 0 ? edge_attr : nullptr;
    a.attr_perm = attr_order == PYG_ORDER_COO ? csr->perm : nullptr;
    a.n_rows = N;
    a.E = E;
    a.msg = msg;
    a.aggr = aggr;
    a.chunk = csr->chunk;
    a.sentinel = E;
    a.out = out;
    a.argmax = argmax;
    a.hint = true;
    return segment_reduce(a, ws, ws_bytes, s);
}

extern "C" int pyg_propagate_heads_workspace(int dtype, int64_t N, int64_t H, int64_t C, int64_t E, int64_t chunk,
                                             size_t *bytes) {
    if (!bytes || !valid_dtype(dtype) || N < 0 || H < 0 || C < 0 || E < 0 || chunk < 0) return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || E >= kMax32 || H * C >= kMax32) return PYG_ERR_UNSUPPORTED;
    *bytes = segment_workspace(E, H * C, PYG_SUM, chunk, N);
    return PYG_OK;
}

extern "C" int pyg_propagate_heads(const void *x, int dtype, int64_t N, int64_t H, int64_t C, const pyg_csr *csr,
                                   const float *alpha, void *out, void *ws, size_t ws_bytes, void *stream) {
    if (!valid_dtype(dtype) || N < 0 || H <= 0 || C < 0 || !csr) return PYG_ERR_INVALID_ARG;
    const int64_t E = csr->E, F = H * C;
    if (N >= kMax32 || E >= kMax32 || F >= kMax32) return PYG_ERR_UNSUPPORTED;
    if (csr->N != N || E < 0 || !csr->rowptr || csr->chunk < 0) return PYG_ERR_INVALID_ARG;
    if (E > 0 && (N == 0 || !csr->col || !alpha)) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && (!x || !out)) return PYG_ERR_INVALID_ARG;
    const int64_t xbytes = N * F * dtype_size(dtype);
    if (overlaps(x, xbytes, out, xbytes) || overlaps(alpha, E * H * 4, out, xbytes)) return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_propagate_heads_workspace(dtype, N, H, C, E, csr->chunk, &need));
    if (ws_bytes < need || (need > 256 && !ws)) return PYG_ERR_WORKSPACE;
    if (N * F == 0) return PYG_OK;
    SegmentArgs a{};
    a.x = x;
    a.dtype = dtype;
    a.F = F;
    a.rowptr = csr->rowptr;
    a.col = csr->col;
    a.alpha = E > 0 ? alpha : nullptr;
    a.H = H;
    a.C = C;
    a.perm = csr->perm;
    a.n_rows = N;
    a.E = E;
    a.msg = PYG_MSG_SRC;
    a.aggr = PYG_SUM;
    a.chunk = csr->chunk;
    a.sentinel = E;
    a.out = out;
    a.hint = true;
    return segment_reduce(a, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

extern "C" int pyg_global_pool_workspace(int dtype, int64_t N, int64_t F, int64_t B, int aggr, size_t *bytes) {
    if (!bytes || !valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || B < 0) return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || B >= kMax32) return PYG_ERR_UNSUPPORTED;
    *bytes = align_up(static_cast<size_t>(B + 1) * sizeof(int64_t), 256) + segment_workspace(N, F, aggr, 0, B);
    return PYG_OK;
}

extern "C" int pyg_global_pool(const void *x, int dtype, int64_t N, int64_t F, const int64_t *batch, int64_t B, int aggr,
                               void *out, int64_t *argmax, void *ws, size_t ws_bytes, void *stream) {
    if (!valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || B < 0) return PYG_ERR_INVALID_ARG;
    if (N >= kMax32 || B >= kMax32) return PYG_ERR_UNSUPPORTED;
    if ((aggr == PYG_MAX) != (argmax != nullptr) && B * F > 0) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_MAX && argmax) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && !x) return PYG_ERR_INVALID_ARG;
    if (B * F > 0 && !out) return PYG_ERR_INVALID_ARG;
    if (N > 0 && (!batch || B == 0)) return PYG_ERR_INVALID_ARG;
    const int64_t esz = dtype_size(dtype);
    if (overlaps(x, N * F * esz, out, B * F * esz)) return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_global_pool_workspace(dtype, N, F, B, aggr, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    if (B * F == 0) return PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    int64_t *ptr = static_cast<int64_t *>(ws);
    const size_t ptr_bytes = align_up(static_cast<size_t>(B + 1) * sizeof(int64_t), 256);
    k_batch_ptr<<<grid_for(B + 1, kBlock), kBlock, 0, s>>>(batch, N, B, ptr);
    PYG_LAUNCH_CHECK();
    SegmentArgs a{};
    a.x = x;
    a.dtype = dtype;
    a.F = F;
    a.rowptr = ptr;
    a.col = nullptr;   // slot n reads node n
    a.weight = nullptr;
    a.perm = nullptr;  // argmax reports the node id
    a.n_rows = B;
    a.E = N;
    a.msg = PYG_MSG_SRC;
    a.aggr = aggr;
    a.chunk = 0;
    a.sentinel = N;
    a.out = out;
    a.argmax = argmax;
    return segment_reduce(a, static_cast<char *>(ws) + ptr_bytes, ws_bytes - ptr_bytes, s);
}

// Edge features of another width D: e = edge_attr Theta_e ([E, D] x [D, F]
// by the dense transform, stored in x's dtype in the workspace), then the
// edge-feature propagate with e. Workspace: e, then the transform's, then the
// propagate's, each 256-byte aligned.
namespace {
struct EncWs {
    size_t e_off, d_off, p_off, bytes;
};
int enc_layout(int dtype, int64_t N, int64_t F, int64_t E, int64_t D, int aggr, int kernel, int64_t chunk, EncWs *w) {
    size_t d = 0, p = 0;
    PYG_TRY(pyg_dense_transform_workspace(D, F, &d));
    PYG_TRY(pyg_propagate_workspace(dtype, N, F, E, aggr, kernel, chunk, &p));
    w->e_off = 0;
    w->d_off = align_up(static_cast<size_t>(E * F * dtype_size(dtype)), 256);
    w->p_off = w->d_off + align_up(d, 256);
    w->bytes = w->p_off + p + 256;
    return PYG_OK;
}
}  // namespace

extern "C" int pyg_propagate_edge_encoded_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t D, int aggr,
                                                    int kernel, int64_t chunk, size_t *bytes) {
    if (!bytes || !valid_dtype(dtype) || !valid_aggr(aggr) || N < 0 || F < 0 || E < 0 || D < 0 || chunk < 0)
        return PYG_ERR_INVALID_ARG;
    EncWs w;
    PYG_TRY(enc_layout(dtype, N, F, E, D, aggr, kernel, chunk, &w));
    *bytes = w.bytes;
    return PYG_OK;
}

extern "C" int pyg_propagate_edge_encoded(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index,
                                          int64_t E, const void *edge_attr, int64_t D, const void *theta_e,
                                          int attr_order, const pyg_csr *csr, int msg, int aggr, int kernel, void *out,
                                          int64_t *argmax, void *ws, size_t ws_bytes, void *stream) {
    if (D < 0) return PYG_ERR_INVALID_ARG;
    bool use_csr = false;  // every check of the edge propagate first: nothing runs before an argument error
    PYG_TRY(check_edge_args(x, dtype, N, F, edge_index, E, edge_attr, E * D * dtype_size(dtype), attr_order, csr,
                            msg, aggr, kernel, out, argmax, &use_csr));
    if (D * F > 0 && !theta_e) return PYG_ERR_INVALID_ARG;
    const int kused = use_csr ? PYG_KERNEL_CSR_SEGMENT : PYG_KERNEL_COO_ATOMIC;
    EncWs w;
    PYG_TRY(enc_layout(dtype, N, F, E, D, aggr, kused, use_csr ? csr->chunk : 0, &w));
    if (!ws || ws_bytes < w.bytes) return PYG_ERR_WORKSPACE;
    char *base = static_cast<char *>(ws);
    void *e = base + w.e_off;
    const int64_t esz = dtype_size(dtype);
    const int64_t wsb = static_cast<int64_t>(ws_bytes);
    if (overlaps(out, N * F * esz, ws, wsb) || overlaps(edge_attr, E * D * esz, ws, wsb) ||
        overlaps(x, N * F * esz, ws, wsb) || overlaps(theta_e, D * F * esz, ws, wsb))
        return PYG_ERR_INVALID_ARG;  // the workspace is written before the inputs are read
    if (E * F > 0) {
        if (D == 0) {  // no edge features: e = 0
            PYG_TRY(fill<uint8_t>(static_cast<uint8_t *>(e), E * F * esz, uint8_t(0), static_cast<hipStream_t>(stream)));
        } else {
            PYG_TRY(pyg_dense_transform(edge_attr, dtype, E, D, theta_e, F, e, dtype, base + w.d_off, w.p_off - w.d_off,
                                        stream));
        }
    }
    return pyg_propagate_edge(x, dtype, N, F, edge_index, E, E * F > 0 ? e : nullptr, attr_order, csr, msg, aggr,
                              kernel, out, argmax, base + w.p_off, ws_bytes - w.p_off, stream);
}
