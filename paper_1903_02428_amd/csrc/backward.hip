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
//
// Edge-feature messages (phi = x_j + e, max(x_j + e, 0), x_j * e) add the
// gradient with respect to the edge features and gate or scale the one with
// respect to x; sum / mean run the segment kernel over the reversed graph
// (edge rows reached through the transpose map or the edge ids), the edge
// gradient is one pass over the CSR slots; max routes as above. fp32 only.
#include "common.hpp"

#ifndef PYG_SDDMM_U
#define PYG_SDDMM_U 4  // slots per sub-group in flight in the weight-gradient dot products
#endif

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

// The same dot products with 16-byte lane vectors (F * sizeof(T) % 16 == 0,
// aligned rows): a sub-group of L = 2^lg lanes covers a feature row (lanes
// loop when it is longer than L vectors), U slots per sub-group in flight;
// the target's gradient row is loaded once per row when one pass covers it.
template <typename T, int U>
__global__ __launch_bounds__(kBlock) void k_sddmm_vec(const T *__restrict__ g, const T *__restrict__ x, int64_t N,
                                                      int64_t F, const int64_t *__restrict__ rowptr,
                                                      const int32_t *__restrict__ col,
                                                      const int64_t *__restrict__ perm, int64_t E, int64_t chunk,
                                                      int lg, int mean, float *__restrict__ grad_w) {
    constexpr int EP = 16 / sizeof(T);
    const int lane = threadIdx.x & (kWave - 1);
    const int L = 1 << lg, S = kWave >> lg;
    const int q = lane & (L - 1), sg = lane >> lg;
    const bool one_pass = F <= (int64_t)L * EP;
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave);
    const int64_t e0 = c * chunk;
    if (e0 >= E) return;
    const int64_t e1 = (e0 + chunk) < E ? (e0 + chunk) : E;
    int64_t r = uniform64(wave_lower_bound(rowptr, N + 1, e0 + 1, lane)) - 1;
    auto dot16 = [](const uint4 &a, const uint4 &b) {
        const uint32_t wa[4] = {a.x, a.y, a.z, a.w}, wb[4] = {b.x, b.y, b.z, b.w};
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (sizeof(T) == 4) {
                acc = fmaf(__uint_as_float(wa[i]), __uint_as_float(wb[i]), acc);
            } else {
                acc = fmaf(__uint_as_float(wa[i] << 16), __uint_as_float(wb[i] << 16), acc);
                acc = fmaf(__uint_as_float(wa[i] & 0xFFFF0000u), __uint_as_float(wb[i] & 0xFFFF0000u), acc);
            }
        }
        return acc;
    };
    while (true) {
        const int64_t s = uniform64(rowptr[r]), t = uniform64(rowptr[r + 1]);
        const int64_t a = s > e0 ? s : e0, b = t < e1 ? t : e1;
        const float sc = mean ? 1.f / static_cast<float>(t - s) : 1.f;
        const int64_t f0 = (int64_t)q * EP;
        uint4 g1 = make_uint4(0, 0, 0, 0);
        if (one_pass && f0 < F && a < b) g1 = *reinterpret_cast<const uint4 *>(g + r * F + f0);
        for (int64_t k0 = a; k0 < b; k0 += (int64_t)S * U) {
            int jj[U];
#pragma unroll
            for (int k = 0; k < U; ++k) {
                const int64_t p = k0 + (int64_t)k * S + sg;
                jj[k] = p < b ? __builtin_nontemporal_load(col + p) : 0;
            }
            float acc[U];
#pragma unroll
            for (int k = 0; k < U; ++k) acc[k] = 0.f;
            for (int64_t f = f0; f < F; f += (int64_t)L * EP) {
                const uint4 gv = one_pass ? g1 : *reinterpret_cast<const uint4 *>(g + r * F + f);
                uint4 xv[U];
#pragma unroll
                for (int k = 0; k < U; ++k) {
                    const int64_t p = k0 + (int64_t)k * S + sg;
                    xv[k] = p < b ? *reinterpret_cast<const uint4 *>(x + (int64_t)jj[k] * F + f) : make_uint4(0, 0, 0, 0);
                }
#pragma unroll
                for (int k = 0; k < U; ++k) acc[k] += dot16(gv, xv[k]);
            }
            for (int off = 1; off < L; off <<= 1)
#pragma unroll
                for (int k = 0; k < U; ++k) acc[k] += __shfl_xor(acc[k], off, kWave);
#pragma unroll
            for (int k = 0; k < U; ++k) {
                const int64_t p = k0 + (int64_t)k * S + sg;
                if (q == 0 && p < b) grad_w[perm[p]] = sc * acc[k];
            }
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
        constexpr int64_t kChunk = 1024;
        const int64_t nchunks = (E + kChunk - 1) / kChunk;
        const unsigned grid = static_cast<unsigned>((nchunks + 3) / 4);
        constexpr int64_t EP = 16 / sizeof(T);
        const bool vec = (F * (int64_t)sizeof(T)) % 16 == 0 && reinterpret_cast<uintptr_t>(g) % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(x) % 16 == 0;
        if (vec && F > 0) {
            int lg = 0;
            while ((int64_t(1) << lg) < F / EP && lg < 6) ++lg;
            k_sddmm_vec<T, PYG_SDDMM_U><<<grid, kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, csr->rowptr, csr->col,
                                                      csr->perm, E, kChunk, lg, aggr == PYG_MEAN, grad_w);
        } else {
            int lg = 0;
            while ((1 << lg) < F && lg < 6) ++lg;
            k_sddmm<T><<<grid, kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, csr->rowptr, csr->col, csr->perm,
                                               E, kChunk, lg, aggr == PYG_MEAN, grad_w);
        }
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}

// grad_e[row(p)] for every CSR slot p = (j -> i): d = gs[i] (the scaled
// upstream gradient), times [x_j + e > 0] (relu) or x_j (mul); the edge row
// is p (CSR order) or perm[p] (COO order). One wavefront per chunk of slots;
// sub-groups of L lanes take one slot each, V floats per lane (V = 4: 16-byte
// vectors when F % 4 == 0 and the arrays are aligned).
template <int V>
__global__ __launch_bounds__(kBlock) void k_edge_grad(const float *__restrict__ gs, const float *__restrict__ x,
                                                      const float *__restrict__ ea, int64_t N, int64_t F,
                                                      const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                                      const int64_t *__restrict__ perm, int64_t E, int64_t chunk, int lg,
                                                      int msg, float *__restrict__ ge) {
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
        for (int64_t p = a + sg; p < b; p += S) {
            const int64_t j = col[p];
            const int64_t er = perm ? perm[p] : p;
            for (int64_t f = (int64_t)q * V; f < F; f += (int64_t)L * V) {
                float d[V], o[V];
                if constexpr (V == 4) {
                    const float4 g4 = *reinterpret_cast<const float4 *>(gs + r * F + f);
                    d[0] = g4.x, d[1] = g4.y, d[2] = g4.z, d[3] = g4.w;
                } else {
                    d[0] = gs[r * F + f];
                }
                if (msg == PYG_MSG_EDGE_ADD) {
#pragma unroll
                    for (int v = 0; v < V; ++v) o[v] = d[v];
                } else {
                    float xv[V], ev[V];
                    if constexpr (V == 4) {
                        const float4 x4 = *reinterpret_cast<const float4 *>(x + j * F + f);
                        xv[0] = x4.x, xv[1] = x4.y, xv[2] = x4.z, xv[3] = x4.w;
                    } else {
                        xv[0] = x[j * F + f];
                    }
                    if (msg == PYG_MSG_EDGE_RELU) {
                        if constexpr (V == 4) {
                            const float4 e4 = *reinterpret_cast<const float4 *>(ea + er * F + f);
                            ev[0] = e4.x, ev[1] = e4.y, ev[2] = e4.z, ev[3] = e4.w;
                        } else {
                            ev[0] = ea[er * F + f];
                        }
#pragma unroll
                        for (int v = 0; v < V; ++v) o[v] = xv[v] + ev[v] > 0.f ? d[v] : 0.f;
                    } else {
#pragma unroll
                        for (int v = 0; v < V; ++v) o[v] = d[v] * xv[v];
                    }
                }
                if constexpr (V == 4)
                    *reinterpret_cast<float4 *>(ge + er * F + f) = make_float4(o[0], o[1], o[2], o[3]);
                else
                    ge[er * F + f] = o[0];
            }
        }
        if (t >= e1) break;
        ++r;
    }
}

// Max: the winning edge k of each output element (i, f) receives g[i, f]:
// grad_x[j, f] += g * dphi/dx (atomics), grad_e[row(k), f] = g * dphi/de (one
// writer per element). Edge rows: k (COO order) or inv[k] (CSR order).
__global__ void k_edge_max_backward(const float *__restrict__ g, const float *__restrict__ x,
                                    const float *__restrict__ ea, int64_t N, int64_t F,
                                    const int64_t *__restrict__ src, int64_t E, const int32_t *__restrict__ inv,
                                    const int64_t *__restrict__ argmax, int msg, float *__restrict__ gx,
                                    float *__restrict__ ge) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < N * F; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = argmax[t];
        if (k < 0 || k >= E) continue;  // empty row (sentinel E)
        const int64_t f = t % F;
        const int64_t j = src[k];
        const int64_t er = inv ? inv[k] : k;
        if (er < 0 || er >= E) continue;  // a malformed permutation: stay in bounds
        const float d = g[t];
        float dx = d, de = d;
        if (msg != PYG_MSG_EDGE_ADD) {
            const float xv = x[j * F + f], ev = ea[er * F + f];
            if (msg == PYG_MSG_EDGE_RELU) {
                const float on = xv + ev > 0.f ? 1.f : 0.f;
                dx = d * on;
                de = d * on;
            } else {
                dx = d * ev;
                de = d * xv;
            }
        }
        if (gx) unsafeAtomicAdd(&gx[j * F + f], dx);
        if (ge) ge[er * F + f] = de;
    }
}

struct EdgeBwdWs {
    float *gs;
    int32_t *inv;
    int32_t *map;
    void *seg;
    size_t seg_bytes;
    size_t bytes;
};

EdgeBwdWs carve_edge_bwd(void *base, int64_t N, int64_t F, int64_t E, int aggr, int64_t chunk_t) {
    Carver c(base);
    EdgeBwdWs w{};
    w.gs = c.take<float>(aggr == PYG_MEAN ? N * F : 0);
    w.inv = c.take<int32_t>(E);
    w.map = c.take<int32_t>(aggr == PYG_MAX ? 0 : E);
    w.seg_bytes = aggr == PYG_MAX ? 0 : segment_workspace(E, F, PYG_SUM, chunk_t, N);
    w.seg = c.take<char>(static_cast<int64_t>(w.seg_bytes));
    w.bytes = c.used + 256;
    return w;
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

extern "C" int pyg_propagate_edge_backward_workspace(int dtype, int64_t N, int64_t F, int64_t E, int aggr,
                                                     int64_t chunk_t, size_t *bytes) {
    if (!bytes || N < 0 || F < 0 || E < 0 || chunk_t < 0) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_SUM && aggr != PYG_MEAN && aggr != PYG_MAX) return PYG_ERR_INVALID_ARG;
    if (dtype == PYG_BF16) return PYG_ERR_UNSUPPORTED;
    if (dtype != PYG_F32) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve_edge_bwd(nullptr, N, F, E, aggr, chunk_t).bytes;
    return PYG_OK;
}

extern "C" int pyg_propagate_edge_backward(const void *grad_out, const void *x, const void *edge_attr, int dtype,
                                           int64_t N, int64_t F, const int64_t *edge_index, const pyg_csr *csr,
                                           const pyg_csr *csr_t, const int32_t *map_t, int attr_order, int msg,
                                           int aggr, const int64_t *argmax, void *grad_x, void *grad_edge_attr,
                                           void *ws, size_t ws_bytes, void *stream) {
    if (dtype == PYG_BF16) return PYG_ERR_UNSUPPORTED;
    if (dtype != PYG_F32 || N < 0 || F < 0 || !csr) return PYG_ERR_INVALID_ARG;
    if (msg != PYG_MSG_EDGE_ADD && msg != PYG_MSG_EDGE_RELU && msg != PYG_MSG_EDGE_MUL) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_SUM && aggr != PYG_MEAN && aggr != PYG_MAX) return PYG_ERR_INVALID_ARG;
    if (attr_order != PYG_ORDER_CSR && attr_order != PYG_ORDER_COO) return PYG_ERR_INVALID_ARG;
    const int64_t E = csr->E;
    if (E < 0 || csr->N != N) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (!grad_x && !grad_edge_attr && (N * F > 0 || E * F > 0)) return PYG_ERR_INVALID_ARG;  // nothing asked for
    if (E > 0 && N == 0) return PYG_ERR_INVALID_ARG;
    if (N * F > 0 && !grad_out) return PYG_ERR_INVALID_ARG;
    if (msg != PYG_MSG_EDGE_ADD && N * F > 0 && (!x || (E * F > 0 && !edge_attr))) return PYG_ERR_INVALID_ARG;
    const bool coo = attr_order == PYG_ORDER_COO;
    const int64_t NF = N * F;
    const float *g = static_cast<const float *>(grad_out);
    const float *xf = static_cast<const float *>(x);
    const float *ea = static_cast<const float *>(edge_attr);
    float *gx = static_cast<float *>(grad_x);
    float *ge = static_cast<float *>(grad_edge_attr);
    int64_t chunk_t = 0;
    if (aggr == PYG_MAX) {
        if (NF > 0 && !argmax) return PYG_ERR_INVALID_ARG;
        if (E > 0 && !edge_index) return PYG_ERR_INVALID_ARG;
        if (E > 0 && !coo && !csr->perm) return PYG_ERR_INVALID_ARG;  // edge id -> CSR slot
    } else {
        if (!csr->rowptr || (E > 0 && !csr->col)) return PYG_ERR_INVALID_ARG;
        if (ge && coo && E > 0 && !csr->perm) return PYG_ERR_INVALID_ARG;
        if (gx) {
            if (!csr_t || csr_t->N != N || csr_t->E != E || !csr_t->rowptr || csr_t->chunk < 0 ||
                (E > 0 && !csr_t->col))
                return PYG_ERR_INVALID_ARG;
            if (msg != PYG_MSG_EDGE_ADD && E > 0) {
                if (coo && !csr_t->perm) return PYG_ERR_INVALID_ARG;
                if (!coo && !map_t && (!csr->perm || !csr_t->perm)) return PYG_ERR_INVALID_ARG;
            }
            chunk_t = csr_t->chunk;
        }
    }
    size_t need;
    PYG_TRY(pyg_propagate_edge_backward_workspace(dtype, N, F, E, aggr, chunk_t, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const EdgeBwdWs w = carve_edge_bwd(ws, N, F, E, aggr, chunk_t);
    if (aggr == PYG_MAX) {
        if (gx) PYG_TRY(fill<float>(gx, NF, 0.f, s));
        if (ge) PYG_TRY(fill<float>(ge, E * F, 0.f, s));
        if (E == 0 || NF == 0) return PYG_OK;
        const int32_t *inv = nullptr;
        if (!coo) {
            PYG_TRY(inverse_perm(csr->perm, E, w.inv, s));
            inv = w.inv;
        }
        k_edge_max_backward<<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, xf, ea, N, F, edge_index, E, inv, argmax,
                                                                       msg, gx, ge);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    if (NF == 0) return PYG_OK;
    // d = s g in fp32 (mean: s_i = 1 / deg_i; sum reads grad_out directly)
    const float *gs = g;
    if (aggr == PYG_MEAN) {
        k_scale_rows<float><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, csr->rowptr, N, F, 1, w.gs);
        PYG_LAUNCH_CHECK();
        gs = w.gs;
    }
    if (gx) {
        SegmentArgs a{};
        a.x = gs;
        a.dtype = PYG_F32;
        a.F = F;
        a.rowptr = csr_t->rowptr;
        a.col = csr_t->col;
        a.n_rows = N;
        a.E = E;
        a.aggr = PYG_SUM;
        a.chunk = csr_t->chunk;
        a.sentinel = E;
        a.out = gx;
        a.hint = true;
        a.msg = PYG_MSG_SRC;  // x_j + e: the scaled gradient of every outgoing edge
        if (msg != PYG_MSG_EDGE_ADD && E > 0) {
            a.msg = msg == PYG_MSG_EDGE_MUL ? PYG_MSG_EDGE_MUL : kSegMsgEdgeReluGrad;
            a.edge_attr = ea;
            a.x_self = xf;
            if (coo) {
                a.attr_perm = csr_t->perm;  // slot q of csr_t is COO edge perm_t[q]
            } else {
                const int32_t *map = map_t;
                if (!map) {
                    PYG_TRY(transpose_map(csr, csr_t, w.inv, w.map, s));
                    map = w.map;
                }
                a.attr_idx = map;
            }
        }
        PYG_TRY(segment_reduce(a, w.seg, w.seg_bytes, s));
    }
    if (ge && E > 0 && F > 0) {
        const bool vec = F % 4 == 0 && reinterpret_cast<uintptr_t>(gs) % 16 == 0 &&
                         (msg == PYG_MSG_EDGE_ADD || reinterpret_cast<uintptr_t>(xf) % 16 == 0) &&
                         (msg != PYG_MSG_EDGE_RELU || reinterpret_cast<uintptr_t>(ea) % 16 == 0) &&
                         reinterpret_cast<uintptr_t>(ge) % 16 == 0;
        const int64_t nv = vec ? F / 4 : F;
        int lg = 0;
        while ((int64_t(1) << lg) < nv && lg < 6) ++lg;
        constexpr int64_t kChunk = 1024;
        const unsigned grid = static_cast<unsigned>(((E + kChunk - 1) / kChunk + 3) / 4);
        const int64_t *perm = coo ? csr->perm : nullptr;
        if (vec)
            k_edge_grad<4><<<grid, kBlock, 0, s>>>(gs, xf, ea, N, F, csr->rowptr, csr->col, perm, E, kChunk, lg, msg, ge);
        else
            k_edge_grad<1><<<grid, kBlock, 0, s>>>(gs, xf, ea, N, F, csr->rowptr, csr->col, perm, E, kChunk, lg, msg, ge);
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}
