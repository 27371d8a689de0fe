// Gradients of the attention path (GAT, an operator of Section 2): the
// multi-head attention sum and the edge scores LeakyReLU(a_src[j] + a_dst[i]).
// (The softmax between them has its own backward in softmax.hip.)
//
// Everything reuses the CSR segment reduction, so every result is
// deterministic:
//   d x       = the attention sum over the reversed graph, with each edge's
//               coefficients moved from its slot in the CSR to its slot in the
//               reversed CSR (the edge id links the two: perm and perm_t);
//   d alpha   = per slot and head, the dot product of the target's upstream
//               gradient block with the source's feature block (C values);
//   d a_dst   = per target, the sum of dL/dv over its CSR row, and
//   d a_src   = per source, the same over its row of the reversed CSR,
//               with dL/dv = dL/de * (v >= 0 ? 1 : slope).
#include "common.hpp"

#include <cmath>

namespace pyg {
namespace {

// inv[perm[p]] = p: the CSR slot of every edge id.
__global__ void k_inverse_perm(const int64_t *__restrict__ perm, int64_t E, int32_t *__restrict__ inv) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < E; p += (int64_t)gridDim.x * blockDim.x)
        inv[perm[p]] = static_cast<int32_t>(p);
}

// out[q, :] = in[inv[perm_t[q]], :] for rows of H floats: values in slot order
// of one CSR, re-ordered into slot order of the reversed CSR.
__global__ void k_to_reversed(const float *__restrict__ in, const int64_t *__restrict__ perm_t,
                              const int32_t *__restrict__ inv, int64_t E, int64_t H, float *__restrict__ out) {
    const int64_t n = E * H;
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t q = t / H, h = t - q * H;
        out[t] = in[(int64_t)inv[perm_t[q]] * H + h];
    }
}

template <typename T>
__device__ __forceinline__ float ldv(const T *p, int64_t i) {
    if constexpr (sizeof(T) == 2) return bf16_bits_to_f32(reinterpret_cast<const uint16_t *>(p)[i]);
    else return p[i];
}

// grad_alpha[p, h] = sum_c g[row(p), h*C + c] * x[col[p], h*C + c]: one
// wavefront per chunk of slots; groups of L lanes take one (slot, head) pair
// and reduce their partial dot products with an xor butterfly.
template <typename T>
__global__ __launch_bounds__(kBlock) void k_head_dots(const T *__restrict__ g, const T *__restrict__ x, int64_t N,
                                                      int64_t H, int64_t C, const int64_t *__restrict__ rowptr,
                                                      const int32_t *__restrict__ col, int64_t E, int64_t chunk,
                                                      int lg, float *__restrict__ grad_alpha) {
    const int lane = threadIdx.x & (kWave - 1);
    const int L = 1 << lg, S = kWave >> lg;
    const int q = lane & (L - 1), sg = lane >> lg;
    const int64_t F = H * C;
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
    const int64_t e0 = c * chunk;
    if (e0 >= E) return;
    const int64_t e1 = (e0 + chunk) < E ? (e0 + chunk) : E;
    int64_t r = uniform64(wave_lower_bound(rowptr, N + 1, e0 + 1, lane)) - 1;  // row holding slot e0
    while (true) {
        const int64_t s = uniform64(rowptr[r]), t = uniform64(rowptr[r + 1]);
        const int64_t a = s > e0 ? s : e0, b = t < e1 ? t : e1;
        const int64_t pairs = (b - a) * H;  // (slot, head) pairs of this row inside the chunk
        for (int64_t k0 = 0; k0 < pairs; k0 += S) {
            const int64_t k = k0 + sg;
            float acc = 0.f;
            int64_t p = 0, h = 0;
            if (k < pairs) {
                p = a + k / H;
                h = k - (k / H) * H;
                const int64_t j = col[p];
                for (int64_t cc = q; cc < C; cc += L) acc = fmaf(ldv(g, r * F + h * C + cc), ldv(x, j * F + h * C + cc), acc);
            }
            for (int off = L >> 1; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
            if (k < pairs && q == 0) grad_alpha[p * H + h] = acc;
        }
        if (t >= e1) break;
        ++r;
    }
}

// dL/dv of every CSR slot: g * (a_src[col] + a_dst[row] >= 0 ? 1 : slope).
__global__ __launch_bounds__(kBlock) void k_gat_dv(const float *__restrict__ a_src, const float *__restrict__ a_dst,
                                                   int64_t N, int64_t H, float slope,
                                                   const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                                   int64_t E, int64_t chunk, const float *__restrict__ g,
                                                   float *__restrict__ dv) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
    const int64_t e0 = c * chunk;
    if (e0 >= E) return;
    const int64_t e1 = (e0 + chunk) < E ? (e0 + chunk) : E;
    int64_t r = uniform64(wave_lower_bound(rowptr, N + 1, e0 + 1, lane)) - 1;
    while (true) {
        const int64_t s = uniform64(rowptr[r]), t = uniform64(rowptr[r + 1]);
        const int64_t a = s > e0 ? s : e0, b = t < e1 ? t : e1;
        for (int64_t k = a * H + lane; k < b * H; k += kWave) {  // (slot, head) elements, contiguous
            const int64_t p = k / H, h = k - p * H;
            const float v = a_src[(int64_t)col[p] * H + h] + a_dst[r * H + h];
            dv[k] = v >= 0.f ? g[k] : slope * g[k];
        }
        if (t >= e1) break;
        ++r;
    }
}

bool csr_ok(const pyg_csr *c, int64_t N, int64_t E) {
    return c && c->N == N && c->E == E && c->rowptr && c->chunk >= 0 && (E == 0 || (c->col && c->perm));
}

struct BwdWs {
    int32_t *inv;
    float *buf_a;
    float *buf_b;
    void *seg;
    size_t seg_bytes;
    size_t bytes;
};

BwdWs carve(void *base, int64_t E, int64_t H, int64_t F_seg, int64_t N, int64_t chunk_t, bool two) {
    Carver c(base);
    BwdWs w{};
    w.inv = c.take<int32_t>(E);
    w.buf_a = c.take<float>(E * H);
    w.buf_b = two ? c.take<float>(E * H) : nullptr;
    w.seg_bytes = segment_workspace(E, F_seg, PYG_SUM, chunk_t, N);
    w.seg = c.take<char>(static_cast<int64_t>(w.seg_bytes));
    w.bytes = c.used + 256;
    return w;
}

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" int pyg_propagate_heads_backward_workspace(int dtype, int64_t N, int64_t H, int64_t C, int64_t E,
                                                      int64_t chunk_t, size_t *bytes) {
    if (!bytes || (dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || H < 0 || C < 0 || E < 0 || chunk_t < 0)
        return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31) || H * C >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve(nullptr, E, H, H * C, N, chunk_t, false).bytes;
    return PYG_OK;
}

extern "C" int pyg_propagate_heads_backward(const void *grad_out, const void *x, int dtype, int64_t N, int64_t H,
                                            int64_t C, const pyg_csr *csr, const pyg_csr *csr_t, const float *alpha,
                                            void *grad_x, float *grad_alpha, void *ws, size_t ws_bytes,
                                            void *stream) {
    if ((dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || H <= 0 || C < 0 || !csr || !csr_t)
        return PYG_ERR_INVALID_ARG;
    const int64_t E = csr->E, F = H * C;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31) || F >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (!csr_ok(csr, N, E) || !csr_ok(csr_t, N, E)) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && !grad_out) return PYG_ERR_INVALID_ARG;
    if (E > 0 && !alpha) return PYG_ERR_INVALID_ARG;
    if (grad_alpha && N * F > 0 && !x) return PYG_ERR_INVALID_ARG;
    if (!grad_x && !grad_alpha) return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_propagate_heads_backward_workspace(dtype, N, H, C, E, csr_t->chunk, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const BwdWs w = carve(ws, E, H, F, N, csr_t->chunk, false);
    if (grad_x && N * F > 0) {
        if (E > 0) {
            k_inverse_perm<<<grid_for(E, kBlock * 4), kBlock, 0, s>>>(csr->perm, E, w.inv);
            PYG_LAUNCH_CHECK();
            k_to_reversed<<<grid_for(E * H, kBlock * 4), kBlock, 0, s>>>(alpha, csr_t->perm, w.inv, E, H, w.buf_a);
            PYG_LAUNCH_CHECK();
        }
        SegmentArgs a{};
        a.x = grad_out;
        a.dtype = dtype;
        a.F = F;
        a.rowptr = csr_t->rowptr;
        a.col = csr_t->col;
        a.alpha = E > 0 ? w.buf_a : nullptr;
        a.H = H;
        a.C = C;
        a.perm = csr_t->perm;
        a.n_rows = N;
        a.E = E;
        a.msg = PYG_MSG_SRC;
        a.aggr = PYG_SUM;
        a.chunk = csr_t->chunk;
        a.sentinel = E;
        a.out = grad_x;
        a.hint = true;
        PYG_TRY(segment_reduce(a, w.seg, w.seg_bytes, s));
    }
    if (grad_alpha && E > 0) {
        int lg = 0;
        while ((1 << lg) < C && lg < 6) ++lg;
        constexpr int64_t kChunk = 1024;
        const int64_t nchunks = (E + kChunk - 1) / kChunk;
        const unsigned grid = static_cast<unsigned>((nchunks + 3) / 4);
        if (dtype == PYG_BF16)
            k_head_dots<uint16_t><<<grid, kBlock, 0, s>>>(static_cast<const uint16_t *>(grad_out),
                                                          static_cast<const uint16_t *>(x), N, H, C, csr->rowptr,
                                                          csr->col, E, kChunk, lg, grad_alpha);
        else
            k_head_dots<float><<<grid, kBlock, 0, s>>>(static_cast<const float *>(grad_out), static_cast<const float *>(x),
                                                       N, H, C, csr->rowptr, csr->col, E, kChunk, lg, grad_alpha);
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}

extern "C" int pyg_gat_scores_backward_workspace(int64_t N, int64_t H, int64_t E, int64_t chunk_t, size_t *bytes) {
    if (!bytes || N < 0 || H < 0 || E < 0 || chunk_t < 0) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    const size_t seg = segment_workspace(E, H, PYG_SUM, 0, N);
    const BwdWs w = carve(nullptr, E, H, H, N, chunk_t, true);
    *bytes = align_up(w.bytes, 256) + seg + 256;
    return PYG_OK;
}

extern "C" int pyg_gat_scores_backward(const float *a_src, const float *a_dst, int64_t H, float negative_slope,
                                       const pyg_csr *csr, const pyg_csr *csr_t, const float *grad_scores,
                                       float *grad_a_src, float *grad_a_dst, void *ws, size_t ws_bytes, void *stream) {
    if (!csr || !csr_t || H <= 0 || !std::isfinite(negative_slope)) return PYG_ERR_INVALID_ARG;
    const int64_t N = csr->N, E = csr->E;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (!csr_ok(csr, N, E) || !csr_ok(csr_t, N, E)) return PYG_ERR_INVALID_ARG;
    if (N * H > 0 && (!a_src || !a_dst || !grad_a_src || !grad_a_dst)) return PYG_ERR_INVALID_ARG;
    if (E > 0 && !grad_scores) return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_gat_scores_backward_workspace(N, H, E, csr_t->chunk, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    if (N * H == 0) return PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const BwdWs w = carve(ws, E, H, H, N, csr_t->chunk, true);
    char *seg_fwd = static_cast<char *>(ws) + align_up(w.bytes, 256);  // workspace of the reduction over csr
    const size_t seg_fwd_bytes = ws_bytes - align_up(w.bytes, 256);
    if (E > 0) {
        constexpr int64_t kChunk = 2048;
        const int64_t nchunks = (E + kChunk - 1) / kChunk;
        k_gat_dv<<<static_cast<unsigned>((nchunks + 3) / 4), kBlock, 0, s>>>(a_src, a_dst, N, H, negative_slope,
                                                                           csr->rowptr, csr->col, E, kChunk,
                                                                           grad_scores, w.buf_a);
        PYG_LAUNCH_CHECK();
        k_inverse_perm<<<grid_for(E, kBlock * 4), kBlock, 0, s>>>(csr->perm, E, w.inv);
        PYG_LAUNCH_CHECK();
        k_to_reversed<<<grid_for(E * H, kBlock * 4), kBlock, 0, s>>>(w.buf_a, csr_t->perm, w.inv, E, H, w.buf_b);
        PYG_LAUNCH_CHECK();
    }
    // d a_dst: rows of csr over the slot-ordered dL/dv; d a_src: rows of csr_t
    for (int side = 0; side < 2; ++side) {
        const pyg_csr *c = side == 0 ? csr : csr_t;
        SegmentArgs a{};
        a.x = side == 0 ? w.buf_a : w.buf_b;
        a.dtype = PYG_F32;
        a.F = H;
        a.rowptr = c->rowptr;
        a.col = nullptr;  // slot p reads row p of dL/dv
        a.n_rows = N;
        a.E = E;
        a.msg = PYG_MSG_SRC;
        a.aggr = PYG_SUM;
        a.chunk = side == 0 ? 0 : c->chunk;
        a.sentinel = E;
        a.out = side == 0 ? static_cast<void *>(grad_a_dst) : static_cast<void *>(grad_a_src);
        PYG_TRY(segment_reduce(a, side == 0 ? static_cast<void *>(seg_fwd) : w.seg,
                               side == 0 ? seg_fwd_bytes : w.seg_bytes, s));
    }
    return PYG_OK;
}
