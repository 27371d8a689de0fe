// Backward of propagate (Eq. (1), gamma = identity) for an upstream gradient
// g = dL/d out:
//   sum / mean  grad_x = the propagate of s*g over the transposed graph,
//               s_i = 1 or 1/deg_i, run by the same segment kernel on the CSR
//               of the reversed edge list (rows = sources) - deterministic;
//               difference messages add the self term -deg_i s_i g_i;
//               grad_w[k] = s_i <g_i, x_j> by a CSR-ordered per-slot dot
//               product (one g row per target row, one x gather per slot),
//               written to COO order through perm - deterministic.
//   max         only the winning edge of each output element receives its
//               gradient: hardware float atomics scatter w_k g into grad_x
//               (and g x_j into grad_w), so sums of colliding winners may
//               differ in the last bits between runs, as Appendix A notes for
//               GPU scatter.
#include "common.hpp"

namespace pyg {
namespace {

template <typename T>
__device__ __forceinline__ float ld(const T *p, int64_t i) {
    if constexpr (sizeof(T) == 2) return bf16_bits_to_f32(reinterpret_cast<const uint16_t *>(p)[i]);
    else return p[i];
}

template <typename T>
__device__ __forceinline__ void st(T *p, int64_t i, float v) {
    if constexpr (sizeof(T) == 2) reinterpret_cast<uint16_t *>(p)[i] = f32_to_bf16_rne(v);
    else p[i] = v;
}

// g'[i,:] = g[i,:] / deg_i (mean; 0 for empty rows) or g[i,:] (sum), in fp32.
template <typename T>
__global__ void k_scale_rows(const T *__restrict__ g, const int64_t *__restrict__ rowptr, int64_t N, int64_t F,
                             int mean, float *__restrict__ out) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < N * F; t += (int64_t)gridDim.x * blockDim.x) {
        if (!mean) {
            out[t] = ld(g, t);
            continue;
        }
        const int64_t i = t / F;
        const int64_t d = rowptr[i + 1] - rowptr[i];
        out[t] = d > 0 ? ld(g, t) / static_cast<float>(d) : 0.f;
    }
}

// Difference messages: grad_x[i,:] -= deg_i * s_i * g[i,:] (sum: s = 1; mean: s = 1/deg), in fp32.
template <typename T>
__global__ void k_diff_self(float *__restrict__ gx, const T *__restrict__ g, const int64_t *__restrict__ rowptr,
                            int64_t N, int64_t F, int mean) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < N * F; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = t / F;
        const int64_t d = rowptr[i + 1] - rowptr[i];
        const float self = mean ? (d > 0 ? ld(g, t) : 0.f) : static_cast<float>(d) * ld(g, t);
        gx[t] -= self;
    }
}

// grad_w[perm[p]] = s_i <g_i, x_{col[p]}> for every slot p of row i: one
// wavefront per chunk of slots; sub-groups of L lanes take one slot each and
// reduce their partial dot products with an xor butterfly.
template <typename T>
__global__ __launch_bounds__(kBlock) void k_sddmm(const T *__restrict__ g, const T *__restrict__ x, int64_t N, int64_t F,
                                                  const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                                  const int64_t *__restrict__ perm, int64_t E, int64_t chunk, int lg,
                                                  int mean, float *__restrict__ grad_w) {
    const int lane = threadIdx.x & (kWave - 1);
    const int L = 1 << lg, S = kWave >> lg;
    const int q = lane & (L - 1), sg = lane >> lg;
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
    const int64_t e0 = c * chunk;
    if (e0 >= E) return;
    const int64_t e1 = (e0 + chunk) < E ? (e0 + chunk) : E;
    int64_t r = uniform64(wave_lower_bound(rowptr, N + 1, e0 + 1, lane)) - 1;  // row holding slot e0
    while (true) {
        const int64_t s = uniform64(rowptr[r]), t = uniform64(rowptr[r + 1]);
        const int64_t a = s > e0 ? s : e0, b = t < e1 ? t : e1;
        const float sc = mean ? 1.f / static_cast<float>(t - s) : 1.f;
        for (int64_t p0 = a; p0 < b; p0 += S) {
            const int64_t p = p0 + sg;
            float acc = 0.f;
            if (p < b) {
                const int64_t j = col[p];
                for (int64_t f = q; f < F; f += L) acc = fmaf(ld(g, r * F + f), ld(x, j * F + f), acc);
            }
            for (int off = L >> 1; off > 0; off >>= 1) acc += __shfl_xor(acc, off, kWave);
            if (p < b && q == 0) grad_w[perm[p]] = sc * acc;
        }
        if (t >= e1) break;
        ++r;
    }
}

// Max: route every output element's gradient to its winning edge.
template <typename T, bool DIFF>
__global__ void k_max_backward(const T *__restrict__ g, const T *__restrict__ x, int64_t N, int64_t F,
                               const int64_t *__restrict__ ei, int64_t E, const float *__restrict__ w,
                               const int64_t *__restrict__ argmax, float *__restrict__ acc, float *__restrict__ grad_w) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < N * F; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = argmax[t];
        if (k < 0 || k >= E) continue;  // empty row (sentinel E)
        const int64_t i = t / F, f = t - i * F;
        const int64_t j = ei[k];
        const float gv = ld(g, t);
        if constexpr (DIFF) {
            unsafeAtomicAdd(&acc[j * F + f], gv);
            unsafeAtomicAdd(&acc[i * F + f], -gv);
        } else {
            unsafeAtomicAdd(&acc[j * F + f], w ? w[k] * gv : gv);
            if (grad_w) unsafeAtomicAdd(&grad_w[k], gv * ld(x, j * F + f));
        }
    }
}

template <typename T>
__global__ void k_cast_out(const float *__restrict__ acc, int64_t n, T *__restrict__ out) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x)
        st(out, t, acc[t]);
}

struct BwdWs {
    void *gscaled;
    float *acc;
    void *seg;
    size_t seg_bytes;
    size_t bytes;
};

// Every intermediate stays in fp32; bf16 gradients are rounded once at the end.
BwdWs carve_bwd(void *base, int dtype, int64_t N, int64_t F, int64_t E, int aggr, int64_t chunk_t) {
    const bool bf16 = dtype == PYG_BF16;
    Carver c(base);
    BwdWs w{};
    w.gscaled = c.take<float>(aggr != PYG_MAX && (aggr == PYG_MEAN || bf16) ? N * F : 0);
    w.acc = c.take<float>(bf16 ? N * F : 0);
    w.seg_bytes = aggr == PYG_MAX ? 0 : segment_workspace(E, F, PYG_SUM, chunk_t, N);
    w.seg = c.take<char>(w.seg_bytes);
    w.bytes = c.used + 256;
    return w;
}

template <typename T>
int backward_typed(const void *grad_out, const void *x, int dtype, int64_t N, int64_t F, const int64_t *ei, int64_t E,
                   const float *ew, const pyg_csr *csr, const pyg_csr *csr_t, int msg, int aggr, const int64_t *argmax,
                   void *grad_x, float *grad_w, const BwdWs &w, hipStream_t s) {
    const T *g = static_cast<const T *>(grad_out);
    const int64_t NF = N * F;
    if (grad_w) PYG_TRY(fill<float>(grad_w, E, 0.f, s));
    if (aggr == PYG_MAX) {
        float *acc = sizeof(T) == 4 ? static_cast<float *>(grad_x) : w.acc;
        PYG_TRY(fill<float>(acc, NF, 0.f, s));
        if (E > 0) {
            if (msg == PYG_MSG_DIFF)
                k_max_backward<T, true><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, ei, E,
                                                                                     ew, argmax, acc, nullptr);
            else
                k_max_backward<T, false><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, ei, E,
                                                                                      ew, argmax, acc, grad_w);
            PYG_LAUNCH_CHECK();
        }
        if (sizeof(T) == 2) {
            k_cast_out<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(acc, NF, static_cast<T *>(grad_x));
            PYG_LAUNCH_CHECK();
        }
        return PYG_OK;
    }
    // g' = s g in fp32 (only fp32 sum can read grad_out directly)
    const bool bf16 = sizeof(T) == 2;
    const float *gs = reinterpret_cast<const float *>(grad_out);
    if (aggr == PYG_MEAN || bf16) {
        k_scale_rows<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, csr ? csr->rowptr : nullptr, N, F,
                                                                    aggr == PYG_MEAN, static_cast<float *>(w.gscaled));
        PYG_LAUNCH_CHECK();
        gs = static_cast<const float *>(w.gscaled);
    }
    float *gx32 = bf16 ? w.acc : static_cast<float *>(grad_x);
    SegmentArgs a{};
    a.x = gs;
    a.dtype = PYG_F32;
    a.F = F;
    a.rowptr = csr_t->rowptr;
    a.col = csr_t->col;
    a.weight = csr_t->weight;
    a.perm = nullptr;
    a.n_rows = N;
    a.E = E;
    a.msg = PYG_MSG_SRC;
    a.aggr = PYG_SUM;
    a.chunk = csr_t->chunk;
    a.sentinel = E;
    a.out = gx32;
    a.argmax = nullptr;
    a.hint = true;
    PYG_TRY(segment_reduce(a, w.seg, w.seg_bytes, s));
    if (msg == PYG_MSG_DIFF) {
        k_diff_self<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(gx32, g, csr->rowptr, N, F, aggr == PYG_MEAN);
        PYG_LAUNCH_CHECK();
    }
    if (bf16) {
        k_cast_out<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(gx32, NF, static_cast<T *>(grad_x));
        PYG_LAUNCH_CHECK();
    }
    if (grad_w && E > 0) {
        int lg = 0;
        while ((1 << lg) < F && lg < 6) ++lg;
        constexpr int64_t kChunk = 1024;
        const int64_t nchunks = (E + kChunk - 1) / kChunk;
        k_sddmm<T><<<static_cast<unsigned>((nchunks + 3) / 4), kBlock, 0, s>>>(
            g, static_cast<const T *>(x), N, F, csr->rowptr, csr->col, csr->perm, E, kChunk, lg, aggr == PYG_MEAN, grad_w);
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}

bool csr_matches(const pyg_csr *c, int64_t N, int64_t E) {
    return c && c->N == N && c->E == E && c->rowptr && (E == 0 || c->col) && c->chunk >= 0;
}

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" int pyg_propagate_backward_workspace(int dtype, int64_t N, int64_t F, int64_t E, int aggr, int64_t chunk_t,
                                                size_t *bytes) {
    if (!bytes || (dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || E < 0 || chunk_t < 0)
        return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_SUM && aggr != PYG_MEAN && aggr != PYG_MAX) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve_bwd(nullptr, dtype, N, F, E, aggr, chunk_t).bytes;
    return PYG_OK;
}

extern "C" int pyg_propagate_backward(const void *grad_out, const void *x, int dtype, int64_t N, int64_t F,
                                      const int64_t *edge_index, int64_t E, const float *edge_weight,
                                      const pyg_csr *csr, const pyg_csr *csr_t, int msg, int aggr,
                                      const int64_t *argmax, void *grad_x, float *grad_w, void *ws, size_t ws_bytes,
                                      void *stream) {
    if ((dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || E < 0) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_SUM && aggr != PYG_MEAN && aggr != PYG_MAX) return PYG_ERR_INVALID_ARG;
    if (msg != PYG_MSG_SRC && msg != PYG_MSG_DIFF) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    const bool weighted = edge_weight != nullptr;
    if (msg == PYG_MSG_DIFF && weighted) return PYG_ERR_INVALID_ARG;
    if (grad_w && (!weighted || msg != PYG_MSG_SRC)) return PYG_ERR_INVALID_ARG;
    if (E > 0 && N == 0) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && (!grad_out || !grad_x)) return PYG_ERR_INVALID_ARG;
    if (grad_w && N * F > 0 && !x) return PYG_ERR_INVALID_ARG;
    const int64_t bytes = N * F * (dtype == PYG_BF16 ? 2 : 4);
    auto overlap = [](const void *a, int64_t an, const void *b, int64_t bn) {
        if (!a || !b || an <= 0 || bn <= 0) return false;
        const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
        return a0 < b0 + bn && b0 < a0 + an;
    };
    if (overlap(grad_x, bytes, grad_out, bytes) || overlap(grad_x, bytes, x, bytes)) return PYG_ERR_INVALID_ARG;
    int64_t chunk_t = 0;
    if (aggr == PYG_MAX) {
        if (N * F > 0 && !argmax) return PYG_ERR_INVALID_ARG;
        if (E > 0 && !edge_index) return PYG_ERR_INVALID_ARG;
    } else {
        if (!csr_matches(csr_t, N, E)) return PYG_ERR_INVALID_ARG;
        if (weighted != (csr_t->weight != nullptr)) return PYG_ERR_INVALID_ARG;
        if ((aggr == PYG_MEAN || msg == PYG_MSG_DIFF || grad_w) && !csr_matches(csr, N, E)) return PYG_ERR_INVALID_ARG;
        if (grad_w && E > 0 && !csr->perm) return PYG_ERR_INVALID_ARG;
        chunk_t = csr_t->chunk;
    }
    const BwdWs w = carve_bwd(ws, dtype, N, F, E, aggr, chunk_t);
    if (ws_bytes < w.bytes || (w.bytes > 256 && !ws)) return PYG_ERR_WORKSPACE;
    if (N * F == 0) return grad_w ? fill<float>(grad_w, E, 0.f, static_cast<hipStream_t>(stream)) : PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dtype == PYG_BF16)
        return backward_typed<uint16_t>(grad_out, x, dtype, N, F, edge_index, E, edge_weight, csr, csr_t, msg, aggr,
                                        argmax, grad_x, grad_w, w, s);
    return backward_typed<float>(grad_out, x, dtype, N, F, edge_index, E, edge_weight, csr, csr_t, msg, aggr, argmax,
                                 grad_x, grad_w, w, s);
}
