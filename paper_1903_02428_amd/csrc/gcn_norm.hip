// GCN edge normalisation (the GCN operator listed in Section 2):
//   d_i = sum_{k: target(k) = i} w_k,  dinv_i = d_i^-1/2 (0 if d_i = 0),
//   norm_k = dinv_j * w_k * dinv_i.
// Unit weights: d is the in-degree from the deterministic LDS histogram.
// Explicit weights: d sums in fp64 hardware atomics. dinv and the edge
// product are fp64, rounded once to fp32 at the end; with unit weights every
// step is order-independent, so the result is reproducible bit for bit.
#include "common.hpp"

#ifndef PYG_NORM_UNROLL
#define PYG_NORM_UNROLL 8  // column loads (then dinv gathers) in flight per lane
#endif
#ifndef PYG_NORM_CHUNK
#define PYG_NORM_CHUNK 2048  // CSR slots per wavefront
#endif

namespace pyg {
namespace {

__global__ void k_weighted_degree(const int64_t *__restrict__ dst, const float *__restrict__ w, int64_t E,
                                  double *__restrict__ d) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < E; k += (int64_t)gridDim.x * blockDim.x)
        unsafeAtomicAdd(&d[dst[k]], w ? static_cast<double>(w[k]) : 1.0);
}

__global__ void k_inv_sqrt(double *__restrict__ d, int64_t N) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x) {
        const double v = d[i];
        d[i] = v > 0.0 ? 1.0 / sqrt(v) : 0.0;
    }
}

// Four edges per thread per iteration keep enough loads in flight.
__global__ __launch_bounds__(kBlock) void k_edge_norm(const int64_t *__restrict__ src, const int64_t *__restrict__ dst,
                                                      const float *__restrict__ w, int64_t E,
                                                      const double *__restrict__ dinv, float *__restrict__ norm) {
    constexpr int U = 4;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (; k + (U - 1) * stride < E; k += U * stride) {
        int64_t j[U], i[U];
        double wk[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            j[u] = src[k + u * stride];
            i[u] = dst[k + u * stride];
            wk[u] = w ? static_cast<double>(w[k + u * stride]) : 1.0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) norm[k + u * stride] = static_cast<float>(dinv[j[u]] * wk[u] * dinv[i[u]]);
    }
    for (; k < E; k += stride) {
        const double wk = w ? static_cast<double>(w[k]) : 1.0;
        norm[k] = static_cast<float>(dinv[src[k]] * wk * dinv[dst[k]]);
    }
}

// ----------------------------------------------------- CSR-ordered variant

// dinv of every row from the row lengths (unit weights).
__global__ void k_row_dinv_count(const int64_t *__restrict__ rowptr, int64_t N, double *__restrict__ dinv) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x) {
        const double d = static_cast<double>(rowptr[i + 1] - rowptr[i]);
        dinv[i] = d > 0.0 ? 1.0 / sqrt(d) : 0.0;
    }
}

// dinv of every row from its CSR-ordered weights: one wavefront per row sums
// in fp64 in a fixed order (lane-strided partial sums, then an xor butterfly).
__global__ __launch_bounds__(kBlock) void k_row_dinv_weighted(const int64_t *__restrict__ rowptr,
                                                              const float *__restrict__ w, int64_t N,
                                                              double *__restrict__ dinv) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t r = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave); r < N; r += waves) {
        const int64_t s = rowptr[r], t = rowptr[r + 1];
        double acc = 0.0;
        for (int64_t p = s + lane; p < t; p += kWave) acc += static_cast<double>(w[p]);
        for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
        if (lane == 0) dinv[r] = acc > 0.0 ? 1.0 / sqrt(acc) : 0.0;
    }
}

// norm_csr[p] = dinv[col[p]] * w[p] * dinv[row(p)]: one wavefront per chunk of
// `chunk` slots; rows crossing chunk edges are simply split (slots are independent).
__global__ __launch_bounds__(kBlock) void k_csr_edge_norm(const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                                          const float *__restrict__ w, int64_t N, int64_t E, int64_t chunk,
                                                          const double *__restrict__ dinv, float *__restrict__ norm) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
    const int64_t e0 = c * chunk;
    if (e0 >= E) return;
    const int64_t e1 = (e0 + chunk) < E ? (e0 + chunk) : E;
    // the row holding slot e0: last row with rowptr[r] <= e0
    int64_t r = uniform64(wave_lower_bound(rowptr, N + 1, e0 + 1, lane)) - 1;
    while (true) {
        const int64_t s = uniform64(rowptr[r]), t = uniform64(rowptr[r + 1]);
        const int64_t a = s > e0 ? s : e0, b = t < e1 ? t : e1;
        const double di = dinv[r];
        // U independent column loads, then U dinv gathers, per lane and batch
        constexpr int U = PYG_NORM_UNROLL;
        for (int64_t p0 = a + lane; p0 < b; p0 += (int64_t)kWave * U) {
            int32_t cj[U];
            float wv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t p = p0 + (int64_t)u * kWave;
                cj[u] = p < b ? col[p] : 0;
                wv[u] = (w && p < b) ? w[p] : 1.f;
            }
            double dj[U];
#pragma unroll
            for (int u = 0; u < U; ++u) dj[u] = p0 + (int64_t)u * kWave < b ? dinv[cj[u]] : 0.0;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t p = p0 + (int64_t)u * kWave;
                if (p < b) norm[p] = static_cast<float>(dj[u] * static_cast<double>(wv[u]) * di);
            }
        }
        if (t >= e1) break;
        r = next_row_with_slots(rowptr, N, r, t, lane);
    }
}

// Short rows (mean degree at most 16): the kernel above walks a chunk's rows
// one after another, a chain of dependent loads per row, which left a
// 13k-edge graph at 360 us. Here the chunks are kNormLightChunk slots and
// lane k of the wavefront takes row r0 + k (the rows that meet the chunk, 64
// at a time) with its slots inside the chunk, so a lane never handles more
// than one chunk of slots, hub rows included. The same expression per slot.
constexpr int64_t kNormLightChunk = 64;
__global__ __launch_bounds__(kBlock) void k_csr_edge_norm_light(const int64_t *__restrict__ rowptr,
                                                                const int32_t *__restrict__ col,
                                                                const float *__restrict__ w, int64_t N, int64_t E,
                                                                const double *__restrict__ dinv,
                                                                float *__restrict__ norm) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
    const int64_t e0 = c * kNormLightChunk;
    if (e0 >= E) return;
    const int64_t e1 = (e0 + kNormLightChunk) < E ? (e0 + kNormLightChunk) : E;
    const int64_t r0 = uniform64(wave_lower_bound(rowptr, N + 1, e0 + 1, lane)) - 1;  // row holding slot e0
    for (int64_t rb = r0;;) {
        const int64_t r = rb + lane;
        if (r < N) {
            const int64_t s = rowptr[r], t = rowptr[r + 1];
            const int64_t a = s > e0 ? s : e0, b = t < e1 ? t : e1;
            if (a < b) {
                const double di = dinv[r];
                for (int64_t p = a; p < b; ++p)
                    norm[p] = static_cast<float>(dinv[col[p]] * static_cast<double>(w ? w[p] : 1.f) * di);
            }
        }
        int64_t nxt = rb + kWave;  // the next batch of rows, if one still starts inside the chunk
        if (nxt >= N) break;
        const int64_t pn = uniform64(rowptr[nxt]);
        if (pn >= e1) break;
        // a whole batch of empty rows ahead (a run of them all starts at pn):
        // go on at the last row that starts at pn
        if (uniform64(rowptr[(nxt + kWave) < N ? (nxt + kWave) : N]) == pn)
            nxt = uniform_lower_bound(rowptr, N + 1, pn + 1) - 1;
        rb = nxt;
    }
}

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" int pyg_gcn_norm_csr_workspace(int64_t N, size_t *bytes) {
    if (N < 0 || !bytes) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = align_up(static_cast<size_t>(N) * sizeof(double), 256) + 256;
    return PYG_OK;
}

extern "C" int pyg_gcn_norm_csr(const pyg_csr *csr, float *norm_csr, void *ws, size_t ws_bytes, void *stream) {
    if (!csr || !csr->rowptr || csr->N < 0 || csr->E < 0) return PYG_ERR_INVALID_ARG;
    const int64_t N = csr->N, E = csr->E;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (E > 0 && (!csr->col || !norm_csr || N == 0)) return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_gcn_norm_csr_workspace(N, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    if (E == 0) return PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    double *dinv = static_cast<double *>(ws);
    if (csr->weight) {
        k_row_dinv_weighted<<<grid_for(N, kBlock / kWave, 1 << 16), kBlock, 0, s>>>(csr->rowptr, csr->weight, N, dinv);
    } else {
        k_row_dinv_count<<<grid_for(N, kBlock * 4), kBlock, 0, s>>>(csr->rowptr, N, dinv);
    }
    PYG_LAUNCH_CHECK();
    if (E <= 16 * N) {  // short rows: a lane per row
        const int64_t nchunks = (E + kNormLightChunk - 1) / kNormLightChunk;
        k_csr_edge_norm_light<<<static_cast<unsigned>((nchunks + 3) / 4), kBlock, 0, s>>>(csr->rowptr, csr->col,
                                                                                        csr->weight, N, E, dinv,
                                                                                        norm_csr);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    constexpr int64_t kChunk = PYG_NORM_CHUNK;
    const int64_t nchunks = (E + kChunk - 1) / kChunk;
    k_csr_edge_norm<<<static_cast<unsigned>((nchunks + 3) / 4), kBlock, 0, s>>>(csr->rowptr, csr->col, csr->weight, N, E,
                                                                              kChunk, dinv, norm_csr);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

extern "C" int pyg_gcn_norm_workspace(int64_t E, int64_t N, size_t *bytes) {
    if (E < 0 || N < 0 || !bytes) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = align_up(static_cast<size_t>(N) * sizeof(double), 256) + degree_workspace(E, N);
    return PYG_OK;
}

__global__ void k_count_to_f64(const int64_t *__restrict__ deg, int64_t N, double *__restrict__ d) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x)
        d[i] = static_cast<double>(deg[i]);
}

extern "C" int pyg_gcn_norm(const int64_t *edge_index, const float *edge_weight, int64_t E, int64_t N,
                            const int64_t *deg, float *norm, void *ws, size_t ws_bytes, void *stream) {
    if (E < 0 || N < 0 || (E > 0 && (!edge_index || !norm || N == 0))) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    size_t need;
    PYG_TRY(pyg_gcn_norm_workspace(E, N, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    if (E == 0) return PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    double *d = static_cast<double *>(ws);
    void *hist_ws = static_cast<char *>(ws) + align_up(static_cast<size_t>(N) * sizeof(double), 256);
    if (edge_weight) {
        PYG_TRY(fill<double>(d, N, 0.0, s));
        k_weighted_degree<<<grid_for(E, kBlock * 8), kBlock, 0, s>>>(edge_index + E, edge_weight, E, d);
        PYG_LAUNCH_CHECK();
    } else if (deg) {  // in-degree already counted (pyg_degree on the same edge list)
        k_count_to_f64<<<grid_for(N, kBlock * 4), kBlock, 0, s>>>(deg, N, d);
        PYG_LAUNCH_CHECK();
    } else {
        PYG_TRY(count_targets_f64(edge_index + E, E, N, d, hist_ws, s));
    }
    k_inv_sqrt<<<grid_for(N, kBlock * 4), kBlock, 0, s>>>(d, N);
    PYG_LAUNCH_CHECK();
    k_edge_norm<<<grid_for(E, kBlock * 4, 1 << 16), kBlock, 0, s>>>(edge_index, edge_index + E, edge_weight, E, d, norm);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

// ---------------------------------------------- normalisation fused into the propagate

extern "C" int pyg_gcn_propagate_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t chunk, size_t *bytes) {
    if (!bytes || (dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || E < 0 || chunk < 0)
        return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    // dinv, the slots' weights (when the caller keeps none), the segment reduction
    *bytes = align_up(static_cast<size_t>(N) * sizeof(double), 256) + align_up(static_cast<size_t>(E) * 4, 256) +
             segment_workspace(E, F, PYG_SUM, chunk, N);
    return PYG_OK;
}

extern "C" int pyg_gcn_propagate(const void *x, int dtype, int64_t N, int64_t F, const pyg_csr *csr, float *norm_out,
                                 void *out, void *ws, size_t ws_bytes, void *stream) {
    if ((dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || !csr || !csr->rowptr) return PYG_ERR_INVALID_ARG;
    const int64_t E = csr->E;
    if (csr->N != N || E < 0 || csr->chunk < 0) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (E > 0 && (!csr->col || N == 0)) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && (!x || !out)) return PYG_ERR_INVALID_ARG;
    const int64_t xbytes = N * F * (dtype == PYG_BF16 ? 2 : 4);
    const uintptr_t xa = reinterpret_cast<uintptr_t>(x), oa = reinterpret_cast<uintptr_t>(out),
                    na = reinterpret_cast<uintptr_t>(norm_out);
    auto overlap = [](uintptr_t a, int64_t an, uintptr_t b, int64_t bn) {
        return a && b && an > 0 && bn > 0 && a < b + static_cast<uintptr_t>(bn) && b < a + static_cast<uintptr_t>(an);
    };
    if (overlap(xa, xbytes, oa, xbytes) || overlap(na, E * 4, xa, xbytes) || overlap(na, E * 4, oa, xbytes))
        return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_gcn_propagate_workspace(dtype, N, F, E, csr->chunk, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    if (N == 0) return PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (F == 0)  // nothing to propagate: the norms alone
        return norm_out ? pyg_gcn_norm_csr(csr, norm_out, ws, ws_bytes, stream) : PYG_OK;
    double *dinv = static_cast<double *>(ws);
    float *norm_ws = reinterpret_cast<float *>(static_cast<char *>(ws) + align_up(static_cast<size_t>(N) * sizeof(double), 256));
    void *seg_ws = reinterpret_cast<char *>(norm_ws) + align_up(static_cast<size_t>(E) * 4, 256);
    if (csr->weight)
        k_row_dinv_weighted<<<grid_for(N, kBlock / kWave, 1 << 16), kBlock, 0, s>>>(csr->rowptr, csr->weight, N, dinv);
    else
        k_row_dinv_count<<<grid_for(N, kBlock * 4), kBlock, 0, s>>>(csr->rowptr, N, dinv);
    PYG_LAUNCH_CHECK();
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
    a.msg = kSegMsgGcn;
    a.aggr = PYG_SUM;
    a.chunk = csr->chunk;
    a.sentinel = E;
    a.out = out;
    a.hint = true;
    a.dinv = dinv;
    a.norm_out = norm_out ? norm_out : norm_ws;  // the later feature windows read the weights back
    return segment_reduce(a, seg_ws, ws_bytes - (static_cast<char *>(seg_ws) - static_cast<char *>(ws)), s);
}

// The norms alone over a source-blocked CSR: one wavefront per virtual row
// b * N + i, d^-1/2 of target i uniform, the same expression per slot.
__global__ __launch_bounds__(kBlock) void k_blocked_slot_norm(const int64_t *__restrict__ brow,
                                                              const int32_t *__restrict__ col,
                                                              const float *__restrict__ w, int64_t N, int64_t B,
                                                              const double *__restrict__ dinv,
                                                              float *__restrict__ norm) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t r = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave); r < B * N; r += waves) {
        const int64_t s = brow[r], t = brow[r + 1];
        const double di = dinv[r % N];
        for (int64_t p = s + lane; p < t; p += kWave) {
            const double wv = w ? static_cast<double>(w[p]) : 1.0;
            norm[p] = static_cast<float>(dinv[col[p]] * wv * di);
        }
    }
}

// Room for the pre-scaled rows d^-1/2 x of the blocked GCN propagate (fp32
// rows: its feature windows after the first gather those, unweighted).
size_t blocked_scaled_bytes(int dtype, int64_t N, int64_t F) {
    return dtype == PYG_F32 ? align_up(static_cast<size_t>(N) * F * 4, 256) : 0;
}

// dinv of every target from a source-blocked CSR: the slots of its B virtual
// rows (unit weights).
__global__ void k_blocked_dinv_count(const int64_t *__restrict__ brow, int64_t N, int64_t B, double *__restrict__ dinv) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t c = 0;
        for (int64_t b = 0; b < B; ++b) c += brow[b * N + i + 1] - brow[b * N + i];
        const double d = static_cast<double>(c);
        dinv[i] = d > 0.0 ? 1.0 / sqrt(d) : 0.0;
    }
}

// ... from its weights: one wavefront per target sums in fp64 over the
// virtual rows in block order (lane-strided partial sums, then an xor
// butterfly): a fixed order.
__global__ __launch_bounds__(kBlock) void k_blocked_dinv_weighted(const int64_t *__restrict__ brow,
                                                                  const float *__restrict__ w, int64_t N, int64_t B,
                                                                  double *__restrict__ dinv) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t i = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave); i < N; i += waves) {
        double acc = 0.0;
        for (int64_t b = 0; b < B; ++b) {
            const int64_t s = brow[b * N + i], t = brow[b * N + i + 1];
            for (int64_t p = s + lane; p < t; p += kWave) acc += static_cast<double>(w[p]);
        }
        for (int off = kWave / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
        if (lane == 0) dinv[i] = acc > 0.0 ? 1.0 / sqrt(acc) : 0.0;
    }
}

// The same over a source-blocked CSR: d and d^-1/2 from the graph's CSR when
// given (its row lengths, or its weights in CSR slot order, exactly as
// above), else from the blocked CSR itself; the propagate over the blocked
// virtual rows, the norms written in the blocked slot order.
extern "C" int pyg_gcn_propagate_blocked_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t B, int64_t chunk,
                                                   size_t *bytes) {
    if (!bytes || (dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || E < 0 || chunk < 0 || B < 2 || B > 32)
        return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = align_up(static_cast<size_t>(N) * sizeof(double), 256) + align_up(static_cast<size_t>(E) * 4, 256) +
             blocked_scaled_bytes(dtype, N, F) + segment_blocked_workspace(E, N, F, B, PYG_SUM, chunk);
    return PYG_OK;
}

extern "C" int pyg_gcn_propagate_blocked(const void *x, int dtype, int64_t N, int64_t F, const pyg_csr *csr,
                                         const pyg_csr_blocks *bcsr, float *norm_out, void *out, void *ws,
                                         size_t ws_bytes, void *stream) {
    if ((dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || !bcsr || !bcsr->rowptr || (csr && !csr->rowptr))
        return PYG_ERR_INVALID_ARG;
    const int64_t E = bcsr->E, B = bcsr->B;
    if (bcsr->N != N || E < 0 || bcsr->chunk < 0 || B < 2 || B > 32) return PYG_ERR_INVALID_ARG;
    if (csr && (csr->N != N || csr->E != E)) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (E > 0 && (!bcsr->col || N == 0)) return PYG_ERR_INVALID_ARG;
    if (csr && (csr->weight != nullptr) != (bcsr->weight != nullptr) && E > 0) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && (!x || !out)) return PYG_ERR_INVALID_ARG;
    const int64_t sz = dtype == PYG_BF16 ? 2 : 4;
    const int64_t xbytes = N * F * sz;
    const uintptr_t xa = reinterpret_cast<uintptr_t>(x), oa = reinterpret_cast<uintptr_t>(out),
                    na = reinterpret_cast<uintptr_t>(norm_out);
    auto overlap = [](uintptr_t a, int64_t an, uintptr_t b, int64_t bn) {
        return a && b && an > 0 && bn > 0 && a < b + static_cast<uintptr_t>(bn) && b < a + static_cast<uintptr_t>(an);
    };
    if (overlap(xa, xbytes, oa, xbytes) || overlap(na, E * 4, xa, xbytes) || overlap(na, E * 4, oa, xbytes))
        return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && ((F * sz) % 16 != 0 || xa % 16 != 0 || oa % 16 != 0)) return PYG_ERR_UNSUPPORTED;
    size_t need;
    PYG_TRY(pyg_gcn_propagate_blocked_workspace(dtype, N, F, E, B, bcsr->chunk, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    if (N == 0) return PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    double *dinv = static_cast<double *>(ws);
    float *norm_ws = reinterpret_cast<float *>(static_cast<char *>(ws) + align_up(static_cast<size_t>(N) * sizeof(double), 256));
    float *xs = reinterpret_cast<float *>(reinterpret_cast<char *>(norm_ws) + align_up(static_cast<size_t>(E) * 4, 256));
    void *seg_ws = reinterpret_cast<char *>(xs) + blocked_scaled_bytes(dtype, N, F);
    if (csr && csr->weight)
        k_row_dinv_weighted<<<grid_for(N, kBlock / kWave, 1 << 16), kBlock, 0, s>>>(csr->rowptr, csr->weight, N, dinv);
    else if (csr)
        k_row_dinv_count<<<grid_for(N, kBlock * 4), kBlock, 0, s>>>(csr->rowptr, N, dinv);
    else if (bcsr->weight)
        k_blocked_dinv_weighted<<<grid_for(N, kBlock / kWave, 1 << 16), kBlock, 0, s>>>(bcsr->rowptr, bcsr->weight, N,
                                                                                      B, dinv);
    else
        k_blocked_dinv_count<<<grid_for(N, kBlock * 4), kBlock, 0, s>>>(bcsr->rowptr, N, B, dinv);
    PYG_LAUNCH_CHECK();
    if (F == 0) {  // nothing to propagate: the norms alone, one slot per lane
        if (!norm_out || E == 0) return PYG_OK;
        k_blocked_slot_norm<<<grid_for(B * N, kBlock / kWave, 1 << 16), kBlock, 0, s>>>(bcsr->rowptr, bcsr->col,
                                                                                      bcsr->weight, N, B, dinv, norm_out);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
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
    a.msg = kSegMsgGcn;
    a.aggr = PYG_SUM;
    a.chunk = bcsr->chunk;
    a.sentinel = E;
    a.out = out;
    a.dinv = dinv;
    a.norm_out = norm_out ? norm_out : norm_ws;  // the later feature windows read the weights back
    a.x_scaled = dtype == PYG_F32 ? xs : nullptr;
    a.norms_wanted = norm_out != nullptr;
    return segment_reduce_blocked(a, B, seg_ws, ws_bytes - (static_cast<char *>(seg_ws) - static_cast<char *>(ws)), s);
}
