// Backward of propagate (Eq. (1), gamma = identity) for an upstream gradient
// g = dL/d out:
//   sum / mean  grad_x = the propagate of s*g over the transposed graph,
//               s_i = 1 or 1/deg_i, run by the same segment kernel on the CSR
//               of the reversed edge list (rows = sources) - deterministic;
//               difference messages add the self term -deg_i s_i g_i;
//               grad_w[k] = s_i <g_i, x_j> by a CSR-ordered per-slot dot
//               product (one g row per target row, one x gather per slot),
//               written in CSR slot order (coalesced) or to COO order
//               through perm (one scattered 4-byte store per edge, about a
//               fifth of the call on the large graph) - deterministic.
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
// gradient is one pass over the CSR slots; max routes as above. fp32 or bf16
// operands; bf16 gradients keep fp32 intermediates and are rounded once.
#include "common.hpp"

#ifndef PYG_SDDMM_U
#define PYG_SDDMM_U 4  // slots per sub-group in flight in the weight-gradient dot products
#endif

namespace pyg {
namespace {

// Slots per wavefront of the kernels that walk a chunk's rows one after
// another (a chain of dependent loads per row): short rows (mean degree at
// most 16) get 64-slot chunks, so the walks are short and the wavefronts
// many; on a 13k-edge graph the 1024-slot chunks left these kernels at
// 130-260 us.
inline int64_t walk_chunk(int64_t E, int64_t N, int64_t dflt) { return E <= 16 * N ? 64 : dflt; }

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

// grad_w[perm[p]] (or grad_w[p] when perm is NULL: CSR order) =
// s_i <g_i, x_{col[p]}> for every slot p of row i: one
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
            if (p < b && q == 0) grad_w[perm ? perm[p] : p] = sc * acc;
        }
        if (t >= e1) break;
        r = next_row_with_slots(rowptr, N, r, t, lane);
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
                if (q == 0 && p < b) grad_w[perm ? perm[p] : p] = sc * acc[k];
            }
        }
        if (t >= e1) break;
        r = next_row_with_slots(rowptr, N, r, t, lane);
    }
}

// Max: route every output element's gradient to its winning edge; grad_w
// entries at the edge id k, or at its CSR slot inv[k] (CSR order).
template <typename T, bool DIFF>
__global__ void k_max_backward(const T *__restrict__ g, const T *__restrict__ x, int64_t N, int64_t F,
                               const int64_t *__restrict__ ei, int64_t E, const float *__restrict__ w,
                               const int64_t *__restrict__ argmax, const int32_t *__restrict__ inv,
                               float *__restrict__ acc, float *__restrict__ grad_w) {
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
            if (grad_w) {
                const int64_t wk = inv ? inv[k] : k;
                if (wk >= 0 && wk < E) unsafeAtomicAdd(&grad_w[wk], gv * ld(x, j * F + f));
            }
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
    int32_t *inv;  // max: slot of every edge id (grad_w in CSR order)
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
    w.inv = c.take<int32_t>(aggr == PYG_MAX ? E : 0);
    w.seg_bytes = aggr == PYG_MAX ? 0 : segment_workspace(E, F, PYG_SUM, chunk_t, N);
    w.seg = c.take<char>(w.seg_bytes);
    w.bytes = c.used + 256;
    return w;
}

template <typename T>
int backward_typed(const void *grad_out, const void *x, int dtype, int64_t N, int64_t F, const int64_t *ei, int64_t E,
                   const float *ew, const pyg_csr *csr, const pyg_csr *csr_t, int msg, int aggr, const int64_t *argmax,
                   void *grad_x, float *grad_w, int w_order, const BwdWs &w, hipStream_t s) {
    const bool w_csr = w_order == PYG_ORDER_CSR;
    const T *g = static_cast<const T *>(grad_out);
    const int64_t NF = N * F;
    if (grad_w) PYG_TRY(fill<float>(grad_w, E, 0.f, s));
    if (aggr == PYG_MAX) {
        float *acc = sizeof(T) == 4 ? static_cast<float *>(grad_x) : w.acc;
        PYG_TRY(fill<float>(acc, NF, 0.f, s));
        if (E > 0) {
            const int32_t *inv = nullptr;
            if (grad_w && w_csr) {
                PYG_TRY(inverse_perm(csr->perm, E, w.inv, s));
                inv = w.inv;
            }
            if (msg == PYG_MSG_DIFF)
                k_max_backward<T, true><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, ei, E,
                                                                                     ew, argmax, nullptr, acc, nullptr);
            else
                k_max_backward<T, false><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, ei, E,
                                                                                      ew, argmax, inv, acc, grad_w);
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
        const int64_t kChunk = walk_chunk(E, N, 1024);
        const int64_t nchunks = (E + kChunk - 1) / kChunk;
        const unsigned grid = static_cast<unsigned>((nchunks + 3) / 4);
        constexpr int64_t EP = 16 / sizeof(T);
        const bool vec = (F * (int64_t)sizeof(T)) % 16 == 0 && reinterpret_cast<uintptr_t>(g) % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(x) % 16 == 0;
        if (vec && F > 0) {
            int lg = 0;
            while ((int64_t(1) << lg) < F / EP && lg < 6) ++lg;
            k_sddmm_vec<T, PYG_SDDMM_U><<<grid, kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, csr->rowptr, csr->col,
                                                      w_csr ? nullptr : csr->perm, E, kChunk, lg, aggr == PYG_MEAN,
                                                      grad_w);
        } else {
            int lg = 0;
            while ((1 << lg) < F && lg < 6) ++lg;
            k_sddmm<T><<<grid, kBlock, 0, s>>>(g, static_cast<const T *>(x), N, F, csr->rowptr, csr->col,
                                               w_csr ? nullptr : csr->perm, E, kChunk, lg, aggr == PYG_MEAN, grad_w);
        }
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}

// V consecutive elements of p as floats / stored from floats: V = 4 is one
// 16-byte fp32 or 8-byte bf16 vector, V = 8 one 16-byte bf16 vector or two
// fp32 ones (the caller checks alignment).
template <typename T, int V>
__device__ __forceinline__ void ldv(const T *p, float (&o)[V]) {
    if constexpr (V == 1) {
        o[0] = ld(p, 0);
    } else if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int h = 0; h < V / 4; ++h) {
            const float4 v = reinterpret_cast<const float4 *>(p)[h];
            o[4 * h] = v.x, o[4 * h + 1] = v.y, o[4 * h + 2] = v.z, o[4 * h + 3] = v.w;
        }
    } else if constexpr (V == 4) {
        const uint2 v = *reinterpret_cast<const uint2 *>(p);
        o[0] = bf16_bits_to_f32(v.x & 0xFFFFu), o[1] = bf16_bits_to_f32(v.x >> 16);
        o[2] = bf16_bits_to_f32(v.y & 0xFFFFu), o[3] = bf16_bits_to_f32(v.y >> 16);
    } else {
        const uint4 v = *reinterpret_cast<const uint4 *>(p);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int h = 0; h < 4; ++h)
            o[2 * h] = bf16_bits_to_f32(w[h] & 0xFFFFu), o[2 * h + 1] = bf16_bits_to_f32(w[h] >> 16);
    }
}

template <typename T, int V>
__device__ __forceinline__ void stv(T *p, const float (&o)[V]) {
    if constexpr (V == 1) {
        st(p, 0, o[0]);
    } else if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int h = 0; h < V / 4; ++h)
            reinterpret_cast<float4 *>(p)[h] = make_float4(o[4 * h], o[4 * h + 1], o[4 * h + 2], o[4 * h + 3]);
    } else {
        uint32_t w[V / 2];
#pragma unroll
        for (int h = 0; h < V / 2; ++h)
            w[h] = uint32_t(f32_to_bf16_rne(o[2 * h])) | (uint32_t(f32_to_bf16_rne(o[2 * h + 1])) << 16);
        if constexpr (V == 4)
            *reinterpret_cast<uint2 *>(p) = make_uint2(w[0], w[1]);
        else
            *reinterpret_cast<uint4 *>(p) = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

// grad_e[row(p)] for every CSR slot p = (j -> i): d = gs[i] (the scaled
// upstream gradient, fp32 or the bf16 gradient itself under sum), times
// [x_j + e > 0] (relu) or x_j (mul), in fp32, rounded once into T; the edge
// row is p (CSR order) or perm[p] (COO order). One wavefront per chunk of
// slots; sub-groups of L lanes take one slot each, V elements per lane
// (V = 4 or 8: vectors when V divides F and the arrays are aligned).
template <typename TG, typename T, int V>
__global__ __launch_bounds__(kBlock) void k_edge_grad(const TG *__restrict__ gs, const T *__restrict__ x,
                                                      const T *__restrict__ ea, int64_t N, int64_t F,
                                                      const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                                      const int64_t *__restrict__ perm, int64_t E, int64_t chunk, int lg,
                                                      int msg, T *__restrict__ ge) {
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
                ldv<TG, V>(gs + r * F + f, d);
                if (msg == PYG_MSG_EDGE_ADD) {
#pragma unroll
                    for (int v = 0; v < V; ++v) o[v] = d[v];
                } else {
                    float xv[V];
                    ldv<T, V>(x + j * F + f, xv);
                    if (msg == PYG_MSG_EDGE_RELU) {
                        float ev[V];
                        ldv<T, V>(ea + er * F + f, ev);
#pragma unroll
                        for (int v = 0; v < V; ++v) o[v] = xv[v] + ev[v] > 0.f ? d[v] : 0.f;
                    } else {
#pragma unroll
                        for (int v = 0; v < V; ++v) o[v] = d[v] * xv[v];
                    }
                }
                stv<T, V>(ge + er * F + f, o);
            }
        }
        if (t >= e1) break;
        r = next_row_with_slots(rowptr, N, r, t, lane);
    }
}

// Max: the winning edge k of each output element (i, f) receives g[i, f]:
// grad_x[j, f] += g * dphi/dx (fp32 atomics into gx), grad_e[row(k), f] =
// g * dphi/de (one writer per element, rounded once into T). Edge rows: k
// (COO order) or inv[k] (CSR order).
template <typename T>
__global__ void k_edge_max_backward(const T *__restrict__ g, const T *__restrict__ x, const T *__restrict__ ea,
                                    int64_t N, int64_t F, const int64_t *__restrict__ src, int64_t E,
                                    const int32_t *__restrict__ inv, const int64_t *__restrict__ argmax, int msg,
                                    float *__restrict__ gx, T *__restrict__ ge) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < N * F; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = argmax[t];
        if (k < 0 || k >= E) continue;  // empty row (sentinel E)
        const int64_t f = t % F;
        const int64_t j = src[k];
        const int64_t er = inv ? inv[k] : k;
        if (er < 0 || er >= E) continue;  // a malformed permutation: stay in bounds
        const float d = ld(g, t);
        float dx = d, de = d;
        if (msg != PYG_MSG_EDGE_ADD) {
            const float xv = ld(x, j * F + f), ev = ld(ea, er * F + f);
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
        if (ge) st(ge, er * F + f, de);
    }
}

// fp32 scratch of the edge-message backward. bf16 keeps every intermediate
// in fp32 and rounds each gradient once: max and mean accumulate grad_x in
// gx32; mean also widens x and the edge rows (relu / mul) so that the
// reversed-graph reduction reads the fp32 scaled gradient beside fp32
// operands. bf16 sum needs none of these: its reduction reads the bf16
// gradient directly and rounds once itself.
struct EdgeBwdWs {
    float *gs;
    float *gx32;
    float *x32;
    float *ea32;
    int32_t *inv;
    int32_t *map;
    void *seg;
    size_t seg_bytes;
    size_t bytes;
};

EdgeBwdWs carve_edge_bwd(void *base, int dtype, int64_t N, int64_t F, int64_t E, int msg, int aggr, int64_t chunk_t) {
    const bool bf16 = dtype == PYG_BF16;
    const bool widen = bf16 && aggr == PYG_MEAN && msg != PYG_MSG_EDGE_ADD;
    Carver c(base);
    EdgeBwdWs w{};
    w.gs = c.take<float>(aggr == PYG_MEAN ? N * F : 0);
    w.gx32 = c.take<float>(bf16 && aggr != PYG_SUM ? N * F : 0);
    w.x32 = c.take<float>(widen ? N * F : 0);
    w.ea32 = c.take<float>(widen ? E * F : 0);
    w.inv = c.take<int32_t>(E);
    w.map = c.take<int32_t>(aggr == PYG_MAX ? 0 : E);
    w.seg_bytes = aggr == PYG_MAX ? 0 : segment_workspace(E, F, PYG_SUM, chunk_t, N);
    w.seg = c.take<char>(static_cast<int64_t>(w.seg_bytes));
    w.bytes = c.used + 256;
    return w;
}

template <typename TG, typename T>
int launch_edge_grad(const TG *gs, const T *x, const T *ea, int64_t N, int64_t F, const pyg_csr *csr,
                     const int64_t *perm, int64_t E, int msg, T *ge, hipStream_t s) {
    // widest vector: 16 bytes of T per lane (4 fp32, 8 bf16)
    const auto fits = [&](int v) {
        const auto al = [](const void *p, size_t b) { return reinterpret_cast<uintptr_t>(p) % b == 0; };
        return F % v == 0 && al(gs, v * sizeof(TG)) && (msg == PYG_MSG_EDGE_ADD || al(x, v * sizeof(T))) &&
               (msg != PYG_MSG_EDGE_RELU || al(ea, v * sizeof(T))) && al(ge, v * sizeof(T));
    };
    const int V = sizeof(T) == 2 && fits(8) ? 8 : fits(4) ? 4 : 1;
    const int64_t nv = F / V;
    int lg = 0;
    while ((int64_t(1) << lg) < nv && lg < 6) ++lg;
    const int64_t kChunk = walk_chunk(E, N, 1024);
    const unsigned grid = static_cast<unsigned>(((E + kChunk - 1) / kChunk + 3) / 4);
    if (V == 8)
        k_edge_grad<TG, T, 8><<<grid, kBlock, 0, s>>>(gs, x, ea, N, F, csr->rowptr, csr->col, perm, E, kChunk, lg,
                                                      msg, ge);
    else if (V == 4)
        k_edge_grad<TG, T, 4><<<grid, kBlock, 0, s>>>(gs, x, ea, N, F, csr->rowptr, csr->col, perm, E, kChunk, lg,
                                                      msg, ge);
    else
        k_edge_grad<TG, T, 1><<<grid, kBlock, 0, s>>>(gs, x, ea, N, F, csr->rowptr, csr->col, perm, E, kChunk, lg,
                                                      msg, ge);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

// Sum / mean / max edge-message backward for T = float or bf16 bits; the
// arguments are checked by the entry point.
template <typename T>
int edge_backward_typed(const T *g, const T *xf, const T *ea, int64_t N, int64_t F, const int64_t *edge_index,
                        const pyg_csr *csr, const pyg_csr *csr_t, const int32_t *map_t, bool coo, int msg, int aggr,
                        const int64_t *argmax, T *gx, T *ge, const EdgeBwdWs &w, hipStream_t s) {
    constexpr bool bf16 = sizeof(T) == 2;
    const int64_t E = csr->E, NF = N * F;
    auto cast_gx = [&](const float *acc) -> int {
        if (!bf16 || !gx || NF == 0) return PYG_OK;
        k_cast_out<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(acc, NF, gx);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    };
    if (aggr == PYG_MAX) {
        float *acc = gx ? (bf16 ? w.gx32 : reinterpret_cast<float *>(gx)) : nullptr;
        if (acc) PYG_TRY(fill<float>(acc, NF, 0.f, s));
        if (ge) PYG_TRY(fill<T>(ge, E * F, T(0), s));  // +0 in fp32 and in bf16 bits
        if (E > 0 && NF > 0) {
            const int32_t *inv = nullptr;
            if (!coo) {
                PYG_TRY(inverse_perm(csr->perm, E, w.inv, s));
                inv = w.inv;
            }
            k_edge_max_backward<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, xf, ea, N, F, edge_index, E, inv,
                                                                              argmax, msg, acc, ge);
            PYG_LAUNCH_CHECK();
        }
        return cast_gx(acc);
    }
    if (NF == 0) return PYG_OK;
    // d = s g in fp32 (mean: s_i = 1 / deg_i); sum reads grad_out directly
    // in its own type (the reductions widen each element as they load it)
    if (aggr == PYG_MEAN) {
        k_scale_rows<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(g, csr->rowptr, N, F, 1, w.gs);
        PYG_LAUNCH_CHECK();
    }
    const bool widen = bf16 && aggr == PYG_MEAN && msg != PYG_MSG_EDGE_ADD;
    if (gx) {
        SegmentArgs a{};
        a.x = aggr == PYG_MEAN ? static_cast<const void *>(w.gs) : static_cast<const void *>(g);
        a.dtype = aggr == PYG_MEAN || !bf16 ? PYG_F32 : PYG_BF16;
        a.F = F;
        a.rowptr = csr_t->rowptr;
        a.col = csr_t->col;
        a.n_rows = N;
        a.E = E;
        a.aggr = PYG_SUM;
        a.chunk = csr_t->chunk;
        a.sentinel = E;
        a.out = bf16 && aggr == PYG_MEAN ? static_cast<void *>(w.gx32) : static_cast<void *>(gx);
        a.hint = true;
        a.msg = PYG_MSG_SRC;  // x_j + e: the scaled gradient of every outgoing edge
        if (msg != PYG_MSG_EDGE_ADD && E > 0) {
            a.msg = msg == PYG_MSG_EDGE_MUL ? PYG_MSG_EDGE_MUL : kSegMsgEdgeReluGrad;
            a.edge_attr = ea;
            a.x_self = xf;
            if (widen) {  // fp32 operands beside the fp32 scaled gradient
                k_scale_rows<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(xf, nullptr, N, F, 0, w.x32);
                PYG_LAUNCH_CHECK();
                k_scale_rows<T><<<grid_for(E * F, kBlock * 4), kBlock, 0, s>>>(ea, nullptr, E, F, 0, w.ea32);
                PYG_LAUNCH_CHECK();
                a.edge_attr = w.ea32;
                a.x_self = w.x32;
            }
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
        if (aggr == PYG_MEAN) PYG_TRY(cast_gx(w.gx32));
    }
    if (ge && E > 0 && F > 0) {
        const int64_t *perm = coo ? csr->perm : nullptr;
        if (aggr == PYG_MEAN || !bf16)
            PYG_TRY((launch_edge_grad<float, T>(aggr == PYG_MEAN ? w.gs : reinterpret_cast<const float *>(g), xf, ea, N,
                                                F, csr, perm, E, msg, ge, s)));
        else
            PYG_TRY((launch_edge_grad<T, T>(g, xf, ea, N, F, csr, perm, E, msg, ge, s)));
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
                                      const int64_t *argmax, void *grad_x, float *grad_w, int w_order, void *ws,
                                      size_t ws_bytes, void *stream) {
    if ((dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || E < 0) return PYG_ERR_INVALID_ARG;
    if (w_order != PYG_ORDER_CSR && w_order != PYG_ORDER_COO) return PYG_ERR_INVALID_ARG;
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
        // grad_w in CSR order: the edge id -> slot map comes from csr->perm
        if (grad_w && w_order == PYG_ORDER_CSR && E > 0 && (!csr_matches(csr, N, E) || !csr->perm))
            return PYG_ERR_INVALID_ARG;
    } else {
        if (!csr_matches(csr_t, N, E)) return PYG_ERR_INVALID_ARG;
        if (weighted != (csr_t->weight != nullptr)) return PYG_ERR_INVALID_ARG;
        if ((aggr == PYG_MEAN || msg == PYG_MSG_DIFF || grad_w) && !csr_matches(csr, N, E)) return PYG_ERR_INVALID_ARG;
        if (grad_w && w_order == PYG_ORDER_COO && E > 0 && !csr->perm) return PYG_ERR_INVALID_ARG;
        chunk_t = csr_t->chunk;
    }
    const BwdWs w = carve_bwd(ws, dtype, N, F, E, aggr, chunk_t);
    if (ws_bytes < w.bytes || (w.bytes > 256 && !ws)) return PYG_ERR_WORKSPACE;
    if (N * F == 0) return grad_w ? fill<float>(grad_w, E, 0.f, static_cast<hipStream_t>(stream)) : PYG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dtype == PYG_BF16)
        return backward_typed<uint16_t>(grad_out, x, dtype, N, F, edge_index, E, edge_weight, csr, csr_t, msg, aggr,
                                        argmax, grad_x, grad_w, w_order, w, s);
    return backward_typed<float>(grad_out, x, dtype, N, F, edge_index, E, edge_weight, csr, csr_t, msg, aggr, argmax,
                                 grad_x, grad_w, w_order, w, s);
}

extern "C" int pyg_propagate_edge_backward_workspace(int dtype, int64_t N, int64_t F, int64_t E, int msg, int aggr,
                                                     int64_t chunk_t, size_t *bytes) {
    if (!bytes || N < 0 || F < 0 || E < 0 || chunk_t < 0) return PYG_ERR_INVALID_ARG;
    if (dtype != PYG_F32 && dtype != PYG_BF16) return PYG_ERR_INVALID_ARG;
    if (msg != PYG_MSG_EDGE_ADD && msg != PYG_MSG_EDGE_RELU && msg != PYG_MSG_EDGE_MUL) return PYG_ERR_INVALID_ARG;
    if (aggr != PYG_SUM && aggr != PYG_MEAN && aggr != PYG_MAX) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve_edge_bwd(nullptr, dtype, N, F, E, msg, aggr, chunk_t).bytes;
    return PYG_OK;
}

extern "C" int pyg_propagate_edge_backward(const void *grad_out, const void *x, const void *edge_attr, int dtype,
                                           int64_t N, int64_t F, const int64_t *edge_index, const pyg_csr *csr,
                                           const pyg_csr *csr_t, const int32_t *map_t, int attr_order, int msg,
                                           int aggr, const int64_t *argmax, void *grad_x, void *grad_edge_attr,
                                           void *ws, size_t ws_bytes, void *stream) {
    if ((dtype != PYG_F32 && dtype != PYG_BF16) || N < 0 || F < 0 || !csr) return PYG_ERR_INVALID_ARG;
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
    int64_t chunk_t = 0;
    if (aggr == PYG_MAX) {
        if (NF > 0 && !argmax) return PYG_ERR_INVALID_ARG;
        if (E > 0 && !edge_index) return PYG_ERR_INVALID_ARG;
        if (E > 0 && !coo && !csr->perm) return PYG_ERR_INVALID_ARG;  // edge id -> CSR slot
    } else {
        if (!csr->rowptr || (E > 0 && !csr->col)) return PYG_ERR_INVALID_ARG;
        if (grad_edge_attr && coo && E > 0 && !csr->perm) return PYG_ERR_INVALID_ARG;
        if (grad_x) {
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
    PYG_TRY(pyg_propagate_edge_backward_workspace(dtype, N, F, E, msg, aggr, chunk_t, &need));
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const EdgeBwdWs w = carve_edge_bwd(ws, dtype, N, F, E, msg, aggr, chunk_t);
    if (dtype == PYG_BF16)
        return edge_backward_typed<uint16_t>(static_cast<const uint16_t *>(grad_out), static_cast<const uint16_t *>(x),
                                             static_cast<const uint16_t *>(edge_attr), N, F, edge_index, csr, csr_t,
                                             map_t, coo, msg, aggr, argmax, static_cast<uint16_t *>(grad_x),
                                             static_cast<uint16_t *>(grad_edge_attr), w, s);
    return edge_backward_typed<float>(static_cast<const float *>(grad_out), static_cast<const float *>(x),
                                      static_cast<const float *>(edge_attr), N, F, edge_index, csr, csr_t, map_t, coo,
                                      msg, aggr, argmax, static_cast<float *>(grad_x),
                                      static_cast<float *>(grad_edge_attr), w, s);
}
