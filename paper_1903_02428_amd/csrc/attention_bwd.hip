// Gradients of the attention path (GAT, an operator of Section 2): the
// multi-head attention sum and the edge scores LeakyReLU(a_src[j] + a_dst[i]).
// (The softmax between them has its own backward in softmax.hip.)
//
// Every sum is a CSR segment reduction in a fixed order, so every result is
// deterministic:
//   d x       = the attention sum over the reversed graph; slot q of the
//               reversed CSR reads its coefficients from row map_t[q] of alpha,
//               the slot of the same edge in the CSR (the transpose map);
//   d alpha   = per slot and head, the dot product of the target's upstream
//               gradient block with the source's feature block (C values);
//   d a_dst   = per target, the sum of dL/dv over its CSR row, and
//   d a_src   = per source, the same over its row of the reversed CSR (rows
//               of dL/dv gathered through map_t),
//               with dL/dv = dL/de * (v >= 0 ? 1 : slope).
#include "common.hpp"

#include <cmath>

namespace pyg {
namespace {

// Slots per wavefront of the kernels that walk a chunk's rows one after
// another (a chain of dependent loads per row): short rows (mean degree at
// most 16) get 64-slot chunks, so the walks are short and the wavefronts
// many; on a 13k-edge graph the 1024-slot chunks left the head dot products
// at 260 us.
inline int64_t walk_chunk(int64_t E, int64_t N, int64_t dflt) { return E <= 16 * N ? 64 : dflt; }

// inv[perm[p]] = p: the CSR slot of every edge id (ids outside [0, E) are
// skipped: a malformed permutation cannot write out of bounds).
__global__ void k_inverse_perm(const int64_t *__restrict__ perm, int64_t E, int32_t *__restrict__ inv) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < E; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = perm[p];
        if (static_cast<uint64_t>(e) < static_cast<uint64_t>(E)) inv[e] = static_cast<int32_t>(p);
    }
}

// map_t[q] = inv[perm_t[q]], clamped into [0, E) so that every consumer's
// reads stay in bounds whatever the permutations hold.
__global__ void k_compose(const int64_t *__restrict__ perm_t, const int32_t *__restrict__ inv, int64_t E,
                          int32_t *__restrict__ map_t) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < E; q += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = perm_t[q];
        int32_t v = static_cast<uint64_t>(e) < static_cast<uint64_t>(E) ? inv[e] : 0;
        map_t[q] = (v >= 0 && v < E) ? v : 0;
    }
}

template <typename T>
__device__ __forceinline__ float ldv(const T *p, int64_t i) {
    if constexpr (sizeof(T) == 2) return bf16_bits_to_f32(reinterpret_cast<const uint16_t *>(p)[i]);
    else return p[i];
}

// grad_alpha[p, h] = sum_c g[row(p), h*C + c] * x[col[p], h*C + c], scalar
// form for any C: one wavefront per chunk of slots; groups of L lanes take
// one (slot, head) pair and reduce their partial dot products with an xor
// butterfly.
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
        r = next_row_with_slots(rowptr, N, r, t, lane);
    }
}

// 16 bytes of T as fp32 values.
template <typename T>
__device__ __forceinline__ void unpack16(const uint4 &u, float (&v)[16 / sizeof(T)]) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = __uint_as_float(w[i]);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
    }
}

// The same dot products with 16-byte lane vectors, the forward's access
// pattern: a sub-group of L = 2^lg lanes covers one window of up to 64 lane
// vectors of a row (features fbase .. fbase + 64 * EP), so each slot costs
// one gathered 16-byte load per lane. The target's gradient row g[r] is read
// once per row and kept in registers; 2^lgh lanes (C / EP, a power of two)
// share a head and reduce with an xor butterfly. U slots per sub-group are in
// flight together, their columns loaded one pass ahead.
template <typename T, int U>
__global__ __launch_bounds__(kBlock) void k_head_dots_vec(const T *__restrict__ g, const T *__restrict__ x, int64_t N,
                                                          int64_t H, int64_t C, int64_t fbase, int64_t nv,
                                                          const int64_t *__restrict__ rowptr,
                                                          const int32_t *__restrict__ col, int64_t E, int64_t chunk,
                                                          int lg, int lgh, float *__restrict__ grad_alpha) {
    constexpr int EP = 16 / sizeof(T);
    const int lane = threadIdx.x & (kWave - 1);
    const int S = kWave >> lg;
    const int q = lane & ((1 << lg) - 1), sg = lane >> lg;
    const int64_t F = H * C;
    const bool act = q < nv;
    const int64_t f0 = fbase + (int64_t)q * EP;
    const int64_t h = act ? f0 / C : 0;
    const bool writer = act && (q & ((1 << lgh) - 1)) == 0;
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
    const int64_t e0 = c * chunk;
    if (e0 >= E) return;
    const int64_t e1 = (e0 + chunk) < E ? (e0 + chunk) : E;
    int64_t r = uniform64(wave_lower_bound(rowptr, N + 1, e0 + 1, lane)) - 1;
    while (true) {
        const int64_t s = uniform64(rowptr[r]), t = uniform64(rowptr[r + 1]);
        const int64_t a = s > e0 ? s : e0, b = t < e1 ? t : e1;
        float gv[EP];
        {
            uint4 u = make_uint4(0, 0, 0, 0);
            if (act && a < b) u = *reinterpret_cast<const uint4 *>(g + r * F + f0);
            unpack16<T>(u, gv);
        }
        int jn[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t p = a + (int64_t)k * S + sg;
            jn[k] = p < b ? __builtin_nontemporal_load(col + p) : 0;
        }
        for (int64_t k0 = a; k0 < b; k0 += (int64_t)S * U) {
            int jj[U];
#pragma unroll
            for (int k = 0; k < U; ++k) jj[k] = jn[k];
#pragma unroll
            for (int k = 0; k < U; ++k) {  // next pass's columns
                const int64_t p = k0 + (int64_t)(U + k) * S + sg;
                jn[k] = p < b ? __builtin_nontemporal_load(col + p) : 0;
            }
            uint4 xv[U];
#pragma unroll
            for (int k = 0; k < U; ++k) {
                const int64_t p = k0 + (int64_t)k * S + sg;
                xv[k] = (act && p < b) ? *reinterpret_cast<const uint4 *>(x + (int64_t)jj[k] * F + f0)
                                       : make_uint4(0, 0, 0, 0);
            }
            float d[U];
#pragma unroll
            for (int k = 0; k < U; ++k) {
                float v[EP];
                unpack16<T>(xv[k], v);
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < EP; ++e) acc = fmaf(gv[e], v[e], acc);
                d[k] = acc;
            }
            for (int off = 1; off < (1 << lgh); off <<= 1)
#pragma unroll
                for (int k = 0; k < U; ++k) d[k] += __shfl_xor(d[k], off, kWave);
#pragma unroll
            for (int k = 0; k < U; ++k) {
                const int64_t p = k0 + (int64_t)k * S + sg;
                if (writer && p < b) grad_alpha[p * H + h] = d[k];
            }
        }
        if (t >= e1) break;
        r = next_row_with_slots(rowptr, N, r, t, lane);
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
        r = next_row_with_slots(rowptr, N, r, t, lane);
    }
}

bool csr_ok(const pyg_csr *c, int64_t N, int64_t E) {
    return c && c->N == N && c->E == E && c->rowptr && c->chunk >= 0 && (E == 0 || (c->col && c->perm));
}


struct BwdWs {
    int32_t *inv;
    int32_t *map;
    float *dv;
    void *seg;
    size_t seg_bytes;
    void *seg2;
    size_t seg2_bytes;
    size_t bytes;
};

// inv and map for a transpose map made on the fly; dv (dL/dv, fp32 [E, H])
// for the score gradient; one segment workspace per reduction.
BwdWs carve(void *base, int64_t E, int64_t H, int64_t F_seg, int64_t N, int64_t chunk_t, bool scores) {
    Carver c(base);
    BwdWs w{};
    w.inv = c.take<int32_t>(E);
    w.map = c.take<int32_t>(E);
    w.dv = scores ? c.take<float>(E * H) : nullptr;
    w.seg_bytes = segment_workspace(E, F_seg, PYG_SUM, chunk_t, N);
    w.seg = c.take<char>(static_cast<int64_t>(w.seg_bytes));
    w.seg2_bytes = scores ? segment_workspace(E, F_seg, PYG_SUM, 0, N) : 0;
    w.seg2 = c.take<char>(static_cast<int64_t>(w.seg2_bytes));
    w.bytes = c.used + 256;
    return w;
}

// Head-dot launch shape: the vector kernel needs 16-byte aligned rows, heads
// made of whole lane vectors, a power-of-two count of them per head and at
// most 64 of them (one wavefront) per head.
template <typename T>
bool head_dots_vec_ok(const void *g, const void *x, int64_t C, int &lgh) {
    constexpr int64_t EP = 16 / sizeof(T);
    if (C <= 0 || C % EP != 0 || reinterpret_cast<uintptr_t>(g) % 16 || reinterpret_cast<uintptr_t>(x) % 16) return false;
    const int64_t lh = C / EP;
    if (lh > kWave || (lh & (lh - 1))) return false;
    lgh = 0;
    while ((int64_t(1) << lgh) < lh) ++lgh;
    return true;
}

template <typename T>
int head_dots(const T *g, const T *x, int64_t N, int64_t H, int64_t C, const pyg_csr *csr, float *grad_alpha,
              hipStream_t s) {
    const int64_t E = csr->E;
    const int64_t kChunk = walk_chunk(E, N, 1024);
    const int64_t nchunks = (E + kChunk - 1) / kChunk;
    const unsigned grid = static_cast<unsigned>((nchunks + 3) / 4);
    int lgh = 0;
    if (head_dots_vec_ok<T>(g, x, C, lgh)) {
        constexpr int64_t EP = 16 / sizeof(T);
        const int64_t nvec = H * C / EP;
        for (int64_t v0 = 0; v0 < nvec; v0 += kWave) {  // windows of 64 lane vectors, whole heads each
            const int64_t nv = (nvec - v0) < kWave ? (nvec - v0) : kWave;
            int lg = 0;
            while ((int64_t(1) << lg) < nv) ++lg;
            k_head_dots_vec<T, 8><<<grid, kBlock, 0, s>>>(g, x, N, H, C, v0 * EP, nv, csr->rowptr, csr->col, E, kChunk,
                                                          lg, lgh, grad_alpha);
            PYG_LAUNCH_CHECK();
        }
        return PYG_OK;
    }
    int lg = 0;
    while ((1 << lg) < C && lg < 6) ++lg;
    k_head_dots<T><<<grid, kBlock, 0, s>>>(g, x, N, H, C, csr->rowptr, csr->col, E, kChunk, lg, grad_alpha);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

}  // namespace

int inverse_perm(const int64_t *perm, int64_t E, int32_t *inv, hipStream_t s) {
    if (E == 0) return PYG_OK;
    k_inverse_perm<<<grid_for(E, kBlock * 4), kBlock, 0, s>>>(perm, E, inv);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

int transpose_map(const pyg_csr *csr, const pyg_csr *csr_t, int32_t *inv, int32_t *map_t, hipStream_t s) {
    const int64_t E = csr->E;
    if (E == 0) return PYG_OK;
    PYG_TRY(inverse_perm(csr->perm, E, inv, s));
    k_compose<<<grid_for(E, kBlock * 4), kBlock, 0, s>>>(csr_t->perm, inv, E, map_t);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

}  // namespace pyg

using namespace pyg;

// Edges from which the map's inverse permutation is partitioned and written
// block by block (inverse_perm_sorted) instead of scattered: below it the
// scattered writes stay in the caches.
constexpr int64_t kInvSortedMin = int64_t(1) << 20;

extern "C" int pyg_csr_transpose_map_workspace(int64_t E, size_t *bytes) {
    if (!bytes || E < 0) return PYG_ERR_INVALID_ARG;
    if (E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = align_up(static_cast<size_t>(E) * sizeof(int32_t), 256) + 256 +
             (E >= kInvSortedMin ? inverse_perm_sorted_workspace(E) : 0);
    return PYG_OK;
}

extern "C" int pyg_csr_transpose_map(const pyg_csr *csr, const pyg_csr *csr_t, int32_t *map_t, void *ws,
                                     size_t ws_bytes, void *stream) {
    if (!csr || !csr_t) return PYG_ERR_INVALID_ARG;
    const int64_t N = csr->N, E = csr->E;
    if (E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (!csr_ok(csr, N, E) || !csr_ok(csr_t, N, E) || (E > 0 && !map_t)) return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_csr_transpose_map_workspace(E, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (E < kInvSortedMin) return transpose_map(csr, csr_t, static_cast<int32_t *>(ws), map_t, s);
    int32_t *inv = static_cast<int32_t *>(ws);
    const size_t inv_bytes = align_up(static_cast<size_t>(E) * sizeof(int32_t), 256);
    PYG_TRY(inverse_perm_sorted(csr->perm, E, inv, static_cast<char *>(ws) + inv_bytes, ws_bytes - inv_bytes, s));
    k_compose<<<grid_for(E, kBlock * 4), kBlock, 0, s>>>(csr_t->perm, inv, E, map_t);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

extern "C" int pyg_propagate_heads_backward_workspace(int dtype, int64_t N, int64_t H, int64_t C, int64_t E,
                                                      int64_t chunk_t, size_t *bytes) {
    if (!bytes || (dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || H < 0 || C < 0 || E < 0 || chunk_t < 0)
        return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31) || H * C >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve(nullptr, E, H, H * C, N, chunk_t, false).bytes;
    return PYG_OK;
}

extern "C" int pyg_propagate_heads_backward(const void *grad_out, const void *x, int dtype, int64_t N, int64_t H,
                                            int64_t C, const pyg_csr *csr, const pyg_csr *csr_t,
                                            const int32_t *map_t, const float *alpha, void *grad_x, float *grad_alpha,
                                            void *ws, size_t ws_bytes, void *stream) {
    if ((dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || H <= 0 || C < 0 || !csr || !csr_t)
        return PYG_ERR_INVALID_ARG;
    const int64_t E = csr->E, F = H * C;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31) || F >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (!csr_ok(csr, N, E) || !csr_ok(csr_t, N, E)) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && !grad_out) return PYG_ERR_INVALID_ARG;
    if (E > 0 && !alpha) return PYG_ERR_INVALID_ARG;
    if (grad_alpha && N * F > 0 && !x) return PYG_ERR_INVALID_ARG;
    if (!grad_x && !grad_alpha && (N * F > 0 || E * H > 0)) return PYG_ERR_INVALID_ARG;  // nothing asked for
    size_t need;
    PYG_TRY(pyg_propagate_heads_backward_workspace(dtype, N, H, C, E, csr_t->chunk, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const BwdWs w = carve(ws, E, H, F, N, csr_t->chunk, false);
    if (grad_x && N * F > 0) {
        const int32_t *map = map_t;
        if (!map && E > 0) {
            PYG_TRY(transpose_map(csr, csr_t, w.inv, w.map, s));
            map = w.map;
        }
        SegmentArgs a{};
        a.x = grad_out;
        a.dtype = dtype;
        a.F = F;
        a.rowptr = csr_t->rowptr;
        a.col = csr_t->col;
        a.alpha = E > 0 ? alpha : nullptr;
        a.alpha_idx = map;
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
    if (grad_alpha && E > 0 && F > 0) {
        if (dtype == PYG_BF16)
            PYG_TRY(head_dots<uint16_t>(static_cast<const uint16_t *>(grad_out), static_cast<const uint16_t *>(x), N,
                                        H, C, csr, grad_alpha, s));
        else
            PYG_TRY(head_dots<float>(static_cast<const float *>(grad_out), static_cast<const float *>(x), N, H, C, csr,
                                     grad_alpha, s));
    } else if (grad_alpha && E > 0) {
        PYG_TRY(fill<float>(grad_alpha, E * H, 0.f, s));  // C = 0: empty dot products
    }
    return PYG_OK;
}

extern "C" int pyg_gat_scores_backward_workspace(int64_t N, int64_t H, int64_t E, int64_t chunk_t, size_t *bytes) {
    if (!bytes || N < 0 || H < 0 || E < 0 || chunk_t < 0) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve(nullptr, E, H, H, N, chunk_t, true).bytes;
    return PYG_OK;
}

extern "C" int pyg_gat_scores_backward(const float *a_src, const float *a_dst, int64_t H, float negative_slope,
                                       const pyg_csr *csr, const pyg_csr *csr_t, const int32_t *map_t,
                                       const float *grad_scores, float *grad_a_src, float *grad_a_dst, void *ws,
                                       size_t ws_bytes, void *stream) {
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
    const int32_t *map = map_t;
    if (E > 0) {
        const int64_t kChunk = walk_chunk(E, N, 2048);
        const int64_t nchunks = (E + kChunk - 1) / kChunk;
        k_gat_dv<<<static_cast<unsigned>((nchunks + 3) / 4), kBlock, 0, s>>>(a_src, a_dst, N, H, negative_slope,
                                                                           csr->rowptr, csr->col, E, kChunk,
                                                                           grad_scores, w.dv);
        PYG_LAUNCH_CHECK();
        if (!map) {
            PYG_TRY(transpose_map(csr, csr_t, w.inv, w.map, s));
            map = w.map;
        }
    }
    // d a_dst: rows of csr over the slot-ordered dL/dv; d a_src: rows of
    // csr_t, slot q reading row map_t[q] of dL/dv
    for (int side = 0; side < 2; ++side) {
        const pyg_csr *c = side == 0 ? csr : csr_t;
        SegmentArgs a{};
        a.x = w.dv;
        a.dtype = PYG_F32;
        a.F = H;
        a.rowptr = c->rowptr;
        a.col = side == 0 ? nullptr : map;  // NULL: slot p reads row p
        a.n_rows = N;
        a.E = E;
        a.msg = PYG_MSG_SRC;
        a.aggr = PYG_SUM;
        a.chunk = side == 0 ? 0 : c->chunk;
        a.sentinel = E;
        a.out = side == 0 ? static_cast<void *>(grad_a_dst) : static_cast<void *>(grad_a_src);
        a.hint = false;  // columns index edges here, not nodes
        PYG_TRY(segment_reduce(a, side == 0 ? w.seg2 : w.seg, side == 0 ? w.seg2_bytes : w.seg_bytes, s));
    }
    return PYG_OK;
}
