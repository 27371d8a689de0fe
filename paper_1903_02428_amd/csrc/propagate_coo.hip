// Gather/scatter over the unsorted COO edge list with hardware atomics: the
// computation scheme of Fig. 1 and Appendix A (gather x_j into edge space,
// form phi, scatter into node space), fused so that no E x F message tensor
// is ever written.
//
//   sum/mean  fp32 global_atomic_add_f32 into an fp32 accumulator (the output
//             itself for fp32 sum, a workspace otherwise), per-target edge
//             counts for mean, then one finalise pass (divide, bf16 round).
//   max       one 64-bit atomic max per element on the key
//             (order_key(phi) << 32) | (0xFFFFFFFF - k): the larger message
//             wins, and among equal messages the smaller edge id k; a decode
//             pass splits the key into the value and the argmax.
//
// Lanes: a group of G = min(64, next_pow2(F)) lanes handles one edge, lane q
// covering features q, q + G, ...; the 64 lanes of a wavefront touch 64
// consecutive floats of a target row per atomic instruction.
#include "common.hpp"

namespace pyg {
namespace {

template <typename T>
__device__ __forceinline__ float load1(const T *p, int64_t i) {
    if constexpr (sizeof(T) == 2) return bf16_bits_to_f32(reinterpret_cast<const uint16_t *>(p)[i]);
    else return p[i];
}

template <typename T>
__device__ __forceinline__ void store1(T *p, int64_t i, float v) {
    if constexpr (sizeof(T) == 2) reinterpret_cast<uint16_t *>(p)[i] = f32_to_bf16_rne(v);
    else p[i] = v;
}

// 0 src, 1 weighted, 2 diff; edge features e_k: 4 x_j + e, 5 max(x_j + e, 0), 6 x_j * e
template <typename T, int MSG>
__device__ __forceinline__ float message(const T *x, int64_t F, int64_t j, int64_t i, int64_t f, float wk,
                                         const T *ea, int64_t k) {
    const float xj = load1(x, j * F + f);
    if constexpr (MSG == 2) return xj - load1(x, i * F + f);
    else if constexpr (MSG == 1) return wk * xj;
    else if constexpr (MSG == 4) return xj + load1(ea, k * F + f);
    else if constexpr (MSG == 5) return (xj + load1(ea, k * F + f)) > 0.f ? (xj + load1(ea, k * F + f)) : 0.f;
    else if constexpr (MSG == 6) return xj * load1(ea, k * F + f);
    else return xj;
}

template <typename T, int MSG, bool COUNT>
__global__ __launch_bounds__(kBlock) void k_coo_add(const T *__restrict__ x, int64_t F, const int64_t *__restrict__ src,
                                                    const int64_t *__restrict__ dst, const float *__restrict__ w,
                                                    const T *__restrict__ ea, int64_t E, int lg,
                                                    float *__restrict__ acc, unsigned *__restrict__ cnt) {
    const int G = 1 << lg;
    const int64_t per_grid = (int64_t)gridDim.x * (kBlock >> lg);
    const int q = threadIdx.x & (G - 1);
    for (int64_t k = (int64_t)blockIdx.x * (kBlock >> lg) + (threadIdx.x >> lg); k < E; k += per_grid) {
        const int64_t j = src[k], i = dst[k];
        const float wk = MSG == 1 ? w[k] : 1.f;
        for (int64_t f = q; f < F; f += G) unsafeAtomicAdd(&acc[i * F + f], message<T, MSG>(x, F, j, i, f, wk, ea, k));
        if (COUNT && q == 0) atomicAdd(&cnt[i], 1u);
    }
}

template <typename T, int MSG>
__global__ __launch_bounds__(kBlock) void k_coo_max(const T *__restrict__ x, int64_t F, const int64_t *__restrict__ src,
                                                    const int64_t *__restrict__ dst, const float *__restrict__ w,
                                                    const T *__restrict__ ea, int64_t E, int lg,
                                                    unsigned long long *__restrict__ keys) {
    const int G = 1 << lg;
    const int64_t per_grid = (int64_t)gridDim.x * (kBlock >> lg);
    const int q = threadIdx.x & (G - 1);
    for (int64_t k = (int64_t)blockIdx.x * (kBlock >> lg) + (threadIdx.x >> lg); k < E; k += per_grid) {
        const int64_t j = src[k], i = dst[k];
        const float wk = MSG == 1 ? w[k] : 1.f;
        const unsigned long long low = 0xFFFFFFFFull - static_cast<unsigned long long>(k);
        for (int64_t f = q; f < F; f += G) {
            const float m = canon_zero(message<T, MSG>(x, F, j, i, f, wk, ea, k));
            atomicMax(&keys[i * F + f], (static_cast<unsigned long long>(order_key(m)) << 32) | low);
        }
    }
}

template <typename T>
__global__ void k_coo_finalize(const float *__restrict__ acc, const unsigned *__restrict__ cnt, int64_t N, int64_t F,
                               T *__restrict__ out) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < N * F; t += (int64_t)gridDim.x * blockDim.x) {
        float v = acc[t];
        if (cnt) {
            const unsigned c = cnt[t / F];
            v = c ? v / static_cast<float>(c) : 0.f;
        }
        store1(out, t, v);
    }
}

template <typename T>
__global__ void k_coo_max_decode(const unsigned long long *__restrict__ keys, int64_t n, int64_t E, T *__restrict__ out,
                                 int64_t *__restrict__ argmax) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) {
        const unsigned long long key = keys[t];
        if (key == 0) {
            store1(out, t, 0.f);
            argmax[t] = E;
        } else {
            store1(out, t, order_key_inv(static_cast<uint32_t>(key >> 32)));
            argmax[t] = static_cast<int64_t>(0xFFFFFFFFull - (key & 0xFFFFFFFFull));
        }
    }
}

template <typename T, int MSG>
int coo_typed(const T *x, int64_t N, int64_t F, const int64_t *ei, int64_t E, const float *w, const T *ea, int aggr,
              T *out, int64_t *argmax, float *acc_ws, unsigned *cnt_ws, unsigned long long *keys_ws, hipStream_t s) {
    int lg = 0;
    while ((1 << lg) < F && lg < 6) ++lg;
    const unsigned grid = grid_for(E, kBlock >> lg, 1 << 18);
    const int64_t NF = N * F;
    if (aggr == PYG_MAX) {
        PYG_TRY(fill<unsigned long long>(keys_ws, NF, 0ull, s));
        if (E > 0) {
            k_coo_max<T, MSG><<<grid, kBlock, 0, s>>>(x, F, ei, ei + E, w, ea, E, lg, keys_ws);
            PYG_LAUNCH_CHECK();
        }
        k_coo_max_decode<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(keys_ws, NF, E, out, argmax);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    const bool direct = sizeof(T) == 4 && aggr == PYG_SUM;  // accumulate straight into out
    float *acc = direct ? reinterpret_cast<float *>(out) : acc_ws;
    unsigned *cnt = aggr == PYG_MEAN ? cnt_ws : nullptr;
    PYG_TRY(fill<float>(acc, NF, 0.f, s));
    if (cnt) PYG_TRY(fill<unsigned>(cnt, N, 0u, s));
    if (E > 0) {
        if (cnt) k_coo_add<T, MSG, true><<<grid, kBlock, 0, s>>>(x, F, ei, ei + E, w, ea, E, lg, acc, cnt);
        else k_coo_add<T, MSG, false><<<grid, kBlock, 0, s>>>(x, F, ei, ei + E, w, ea, E, lg, acc, nullptr);
        PYG_LAUNCH_CHECK();
    }
    if (!direct) {
        k_coo_finalize<T><<<grid_for(NF, kBlock * 4), kBlock, 0, s>>>(acc, cnt, N, F, out);
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}

template <typename T>
int coo_msg(const T *x, int64_t N, int64_t F, const int64_t *ei, int64_t E, const float *w, const T *ea, int msg,
            int aggr, T *out, int64_t *argmax, float *acc_ws, unsigned *cnt_ws, unsigned long long *keys_ws,
            hipStream_t s) {
#define PYG_COO_CASE(K) return coo_typed<T, K>(x, N, F, ei, E, w, ea, aggr, out, argmax, acc_ws, cnt_ws, keys_ws, s)
    if (msg == PYG_MSG_DIFF) PYG_COO_CASE(2);
    if (msg == PYG_MSG_EDGE_ADD) PYG_COO_CASE(4);
    if (msg == PYG_MSG_EDGE_RELU) PYG_COO_CASE(5);
    if (msg == PYG_MSG_EDGE_MUL) PYG_COO_CASE(6);
    if (w) PYG_COO_CASE(1);
    PYG_COO_CASE(0);
#undef PYG_COO_CASE
}

}  // namespace

struct CooWs {
    float *acc;
    unsigned *cnt;
    unsigned long long *keys;
    size_t bytes;
};

static CooWs carve_coo(void *base, int dtype, int64_t N, int64_t F, int aggr) {
    Carver c(base);
    CooWs w{};
    const bool need_acc = aggr != PYG_MAX && !(dtype == PYG_F32 && aggr == PYG_SUM);
    w.acc = c.take<float>(need_acc ? N * F : 0);
    w.cnt = c.take<unsigned>(aggr == PYG_MEAN ? N : 0);
    w.keys = c.take<unsigned long long>(aggr == PYG_MAX ? N * F : 0);
    w.bytes = c.used + 256;
    return w;
}

size_t coo_workspace(int dtype, int64_t N, int64_t F, int aggr) { return carve_coo(nullptr, dtype, N, F, aggr).bytes; }

int coo_propagate(const void *x, int dtype, int64_t N, int64_t F, const int64_t *ei, int64_t E, const float *w, int msg,
                  int aggr, void *out, int64_t *argmax, void *ws, size_t ws_bytes, hipStream_t s, const void *ea) {
    const CooWs cw = carve_coo(ws, dtype, N, F, aggr);
    if (ws_bytes < cw.bytes || (cw.bytes > 256 && !ws)) return PYG_ERR_WORKSPACE;
    if (dtype == PYG_BF16)
        return coo_msg<uint16_t>(static_cast<const uint16_t *>(x), N, F, ei, E, w, static_cast<const uint16_t *>(ea),
                                 msg, aggr, static_cast<uint16_t *>(out), argmax, cw.acc, cw.cnt, cw.keys, s);
    return coo_msg<float>(static_cast<const float *>(x), N, F, ei, E, w, static_cast<const float *>(ea), msg, aggr,
                          static_cast<float *>(out), argmax, cw.acc, cw.cnt, cw.keys, s);
}

}  // namespace pyg
