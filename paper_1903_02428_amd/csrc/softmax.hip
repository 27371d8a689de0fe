// Softmax over the incoming edges of every target, per attention head (the
// normalisation of GAT's attention coefficients; Section 3 attributes GAT's
// runtime to a dedicated sparse softmax), its backward, and the fused form
// that computes GAT's edge scores LeakyReLU(a_src[j] + a_dst[i]) on the fly.
//
// Data: every edge carries H fp32 values, row-major [E,H]. They are read and
// written either in CSR slot order (coalesced) or in COO edge order through
// csr->perm.
//
// Work split, as in the propagate kernel: E slots cut into chunks, one
// wavefront per chunk. A row of at most `chunk` slots belongs to the chunk
// holding its first slot and is done there by a group of G lanes (short
// rows share a wavefront when the mean degree is small).
// Vector path (H a power of two, 16-byte aligned arrays): a row's values are
// the flat range [s*H, t*H) of the [E,H] array and each lane takes 16-byte
// blocks of it, so a lane's four elements always belong to the same four
// heads (H >= 4) or repeat the heads (H = 1, 2). A row that fits the group's
// registers (R blocks per lane) is read once: maximum, then exp and sum with
// the exponentials kept in registers, then scaled stores. A larger row makes
// an online pass (per-batch maximum, one exp per element, rescaling the sum)
// and a second pass that recomputes and stores.
// Scalar path (any H): Hq lanes (H rounded up to a power of two, at most 64)
// cover the heads of one slot, G / Hq slots go side by side; online pass,
// then normalising pass.
// A longer row is cut at chunk boundaries: every piece's (max, sum) goes to
// a partial, a fold kernel merges the partials of each long row in chunk
// order, and a third kernel normalises the pieces. All orders are fixed, so
// results are bit-reproducible.
#include "common.hpp"

#include <math.h>

// 16-byte blocks per lane held in registers by the vector path (forward,
// backward); a row of up to G * R blocks is read once.
#ifndef PYG_SOFTMAX_REGS
#define PYG_SOFTMAX_REGS 8
#endif
#ifndef PYG_SOFTMAX_REGS_BWD
#define PYG_SOFTMAX_REGS_BWD 8
#endif
// 16-byte blocks per lane and batch of the two-pass path (rows too large for
// registers, and long-row pieces)
#ifndef PYG_SOFTMAX_STREAM
#define PYG_SOFTMAX_STREAM 8
#endif

namespace pyg {
namespace {

constexpr int kScores = 0, kGat = 1, kBackward = 2;

struct SmParams {
    const float *s;       // scores (kScores) or alpha (kBackward), [E,H]
    const float *g;       // dL/d alpha (kBackward), [E,H]
    const float *a_src;   // kGat: [N,H]
    const float *a_dst;   // kGat: [N,H]
    float slope;
    const int64_t *rowptr;
    const int32_t *col;
    const int64_t *perm;  // non-NULL: per-edge arrays are indexed by COO edge id perm[slot]
    int64_t n_rows;
    int64_t E;
    int64_t H;
    int64_t chunk;
    int64_t nchunks;
    int lg_h;   // scalar path: log2 of lanes per slot (Hq)
    int lg_hh;  // vector path: log2 of H
    int lg_g;   // log2 of lanes per short row
    float *out;
    float2 *part;       // [2 * nchunks, H]: piece states (continuing piece at 2c, head piece at 2c + 1)
    float2 *stat;       // [nchunks, H]: folded state of the long row that starts in chunk c
    int32_t *head_row;  // [nchunks]: long row starting in chunk c, or -1
    int32_t *cont_row;  // [nchunks]: long row continuing into chunk c, or -1
};

// exp(x) on the hardware exp2 unit as 2^(x log2 e): rounding the product
// changes the result by at most |x| eps relative, the unit adds about one
// ulp. It is only called on finite arguments: padding (-inf) and empty
// states are mapped to 0 by explicit selects (pexp), which also keeps the
// result independent of how the compiler treats exp2 of -inf.
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }
__device__ __forceinline__ float pexp(float v, float m) { return v == -INFINITY ? 0.f : fexp(v - m); }

// Running state of one (row, head): forward (m = max, d = sum exp(v - m)),
// backward (m = sum alpha * g, d unused).
template <int SRC>
__device__ __forceinline__ void merge(float &m, float &d, float m2, float d2) {
    if constexpr (SRC == kBackward) {
        m += m2;
    } else {
        if (m2 > m) {
            d = pexp(m, m2) * d + d2;
            m = m2;
        } else if (m2 != -INFINITY) {
            d += d2 * fexp(m2 - m);
        }
    }
}

template <int SRC>
__device__ __forceinline__ float2 identity_state() {
    return SRC == kBackward ? make_float2(0.f, 0.f) : make_float2(-INFINITY, 0.f);
}

__device__ __forceinline__ int64_t edge_of(const SmParams &p, int64_t slot) { return p.perm ? p.perm[slot] : slot; }

// Value of slot `slot`, head h: the score (forward) or alpha (backward, with
// the upstream gradient in *gv). adst is a_dst[row, h] for kGat.
template <int SRC>
__device__ __forceinline__ float value(const SmParams &p, int64_t slot, int64_t h, float adst, float *gv) {
    if constexpr (SRC == kGat) {
        const float v = p.a_src[(int64_t)p.col[slot] * p.H + h] + adst;
        return v >= 0.f ? v : p.slope * v;
    } else {
        const int64_t e = edge_of(p, slot) * p.H + h;
        if constexpr (SRC == kBackward) *gv = p.g[e];
        return p.s[e];
    }
}

template <int SRC>
__device__ __forceinline__ void accumulate(float &m, float &d, float v, float gv) {
    if constexpr (SRC == kBackward) {
        m = fmaf(v, gv, m);
    } else if (v > m) {
        d = pexp(m, v) * d + 1.f;
        m = v;
    } else {
        d += fexp(v - m);
    }
}

// State of slots [s, t) of row r for head block hb over a group of 2^lg_g
// lanes (l = lane within the group). Every lane of a head ends with the
// group's state (the butterfly is symmetric).
template <int SRC>
__device__ __forceinline__ float2 row_state(const SmParams &p, int64_t r, int64_t s, int64_t t, int64_t hb, int lg_g,
                                            int l) {
    constexpr int U = 4;
    const int64_t h = hb + (l & ((1 << p.lg_h) - 1));
    const int step = 1 << (lg_g - p.lg_h);
    const bool on = h < p.H;
    const float adst = (SRC == kGat && on) ? p.a_dst[r * p.H + h] : 0.f;
    float2 st = identity_state<SRC>();
    if (on) {
        for (int64_t b = s + (l >> p.lg_h); b < t; b += (int64_t)U * step) {
            float v[U], gv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t q = b + (int64_t)u * step;
                gv[u] = 0.f;
                v[u] = q < t ? value<SRC>(p, q, h, adst, &gv[u]) : 0.f;
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (b + (int64_t)u * step < t) accumulate<SRC>(st.x, st.y, v[u], gv[u]);
        }
    }
    for (int off = 1 << p.lg_h; off < (1 << lg_g); off <<= 1) {
        const float m2 = __shfl_xor(st.x, off, kWave);
        const float d2 = __shfl_xor(st.y, off, kWave);
        merge<SRC>(st.x, st.y, m2, d2);
    }
    return st;
}

// Write the outputs of slots [s, t) of row r for head block hb from the
// row's final state.
template <int SRC>
__device__ __forceinline__ void row_write(const SmParams &p, int64_t r, int64_t s, int64_t t, int64_t hb, int lg_g,
                                          int l, float2 st) {
    constexpr int U = 4;
    const int64_t h = hb + (l & ((1 << p.lg_h) - 1));
    if (h >= p.H) return;
    const int step = 1 << (lg_g - p.lg_h);
    const float adst = SRC == kGat ? p.a_dst[r * p.H + h] : 0.f;
    const float inv = SRC == kBackward ? 0.f : 1.f / st.y;
    for (int64_t b = s + (l >> p.lg_h); b < t; b += (int64_t)U * step) {
        float v[U], gv[U];
        int64_t e[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t q = b + (int64_t)u * step;
            gv[u] = 0.f;
            v[u] = q < t ? value<SRC>(p, q, h, adst, &gv[u]) : 0.f;
            e[u] = q < t ? edge_of(p, q) * p.H + h : -1;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (e[u] < 0) continue;
            if constexpr (SRC == kBackward) p.out[e[u]] = v[u] * (gv[u] - st.x);
            else p.out[e[u]] = fexp(v[u] - st.x) * inv;
        }
    }
}

// State of a piece of a long row over the whole wavefront, stored as a partial.
template <int SRC>
__device__ __forceinline__ void piece_state(const SmParams &p, int64_t r, int64_t s, int64_t t, int64_t slot, int lane) {
    for (int64_t hb = 0; hb < p.H; hb += (1 << p.lg_h)) {
        const float2 st = row_state<SRC>(p, r, s, t, hb, 6, lane);
        const int64_t h = hb + (lane & ((1 << p.lg_h) - 1));
        if ((lane >> p.lg_h) == 0 && h < p.H) p.part[slot * p.H + h] = st;
    }
}

// ------------------------------------------------------------ vector path
template <int SRC>
__device__ __forceinline__ float pad_value() { return SRC == kBackward ? 0.f : -INFINITY; }

__device__ __forceinline__ float leaky(float v, float slope) { return v >= 0.f ? v : slope * v; }

// Block b of the flat [E,H] range of a row (elements 4b .. 4b+3, those
// outside [lo, hi) padded). H >= 4: one slot, heads (4b mod H) + i, the row
// covers whole blocks. H < 4: slots (4b + i) / H, heads i mod H.
template <int SRC, int VH>
__device__ __forceinline__ void vload(const SmParams &p, int64_t b, int64_t lo, int64_t hi, const float (&adst)[4],
                                      float (&v)[4], float (&gv)[4]) {
    const int64_t f = 4 * b;
    if constexpr (VH == 4) {
        const int64_t slot = f >> p.lg_hh;
        const int64_t j = f & (p.H - 1);
        if constexpr (SRC == kGat) {
            const float4 a = *reinterpret_cast<const float4 *>(p.a_src + (int64_t)p.col[slot] * p.H + j);
            v[0] = leaky(a.x + adst[0], p.slope);
            v[1] = leaky(a.y + adst[1], p.slope);
            v[2] = leaky(a.z + adst[2], p.slope);
            v[3] = leaky(a.w + adst[3], p.slope);
        } else {
            const int64_t e = p.perm ? p.perm[slot] * p.H + j : f;  // CSR order: slot * H + j = f
            const float4 a = *reinterpret_cast<const float4 *>(p.s + e);
            v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w;
            if constexpr (SRC == kBackward) {
                const float4 q = *reinterpret_cast<const float4 *>(p.g + e);
                gv[0] = q.x, gv[1] = q.y, gv[2] = q.z, gv[3] = q.w;
            }
        }
        return;
    } else {
    if (SRC != kGat && !p.perm && f >= lo && f + 4 <= hi) {
        const float4 a = *reinterpret_cast<const float4 *>(p.s + f);
        v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w;
        if constexpr (SRC == kBackward) {
            const float4 q = *reinterpret_cast<const float4 *>(p.g + f);
            gv[0] = q.x, gv[1] = q.y, gv[2] = q.z, gv[3] = q.w;
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t fi = f + i;
        v[i] = pad_value<SRC>();
        gv[i] = 0.f;
        if (fi < lo || fi >= hi) continue;
        const int64_t slot = fi >> p.lg_hh;
        const int64_t h = fi & (p.H - 1);
        if constexpr (SRC == kGat) {
            v[i] = leaky(p.a_src[(int64_t)p.col[slot] * p.H + h] + adst[i], p.slope);
        } else {
            const int64_t e = (p.perm ? p.perm[slot] : slot) * p.H + h;
            v[i] = p.s[e];
            if constexpr (SRC == kBackward) gv[i] = p.g[e];
        }
    }
    }
}

// Store block b of the row's outputs (elements inside [lo, hi) only).
template <int VH>
__device__ __forceinline__ void vstore(const SmParams &p, int64_t b, int64_t lo, int64_t hi, const float (&o)[4]) {
    const int64_t f = 4 * b;
    if constexpr (VH == 4) {
        const int64_t e = p.perm ? p.perm[f >> p.lg_hh] * p.H + (f & (p.H - 1)) : f;
        *reinterpret_cast<float4 *>(p.out + e) = make_float4(o[0], o[1], o[2], o[3]);
        return;
    }
    if (!p.perm && f >= lo && f + 4 <= hi) {
        *reinterpret_cast<float4 *>(p.out + f) = make_float4(o[0], o[1], o[2], o[3]);
        return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t fi = f + i;
        if (fi < lo || fi >= hi) continue;
        const int64_t slot = fi >> p.lg_hh;
        p.out[(p.perm ? p.perm[slot] : slot) * p.H + (fi & (p.H - 1))] = o[i];
    }
}

// Combine per-element values over everything that shares a head: the other
// elements of the lane (H = 1, 2), then lanes H/4 apart inside the group.
template <int VH, typename OP>
__device__ __forceinline__ void vcombine(const SmParams &p, int G, float (&x)[4], OP op) {
    if constexpr (VH == 1) {
        const float a = op(op(x[0], x[1]), op(x[2], x[3]));
        x[0] = x[1] = x[2] = x[3] = a;
    } else if constexpr (VH == 2) {
        x[0] = x[2] = op(x[0], x[2]);
        x[1] = x[3] = op(x[1], x[3]);
    }
    for (int off = VH == 4 ? static_cast<int>(p.H >> 2) : 1; off < G; off <<= 1)
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = op(x[i], __shfl_xor(x[i], off, kWave));
}

// Same for (max, sum) states of the forward.
template <int VH>
__device__ __forceinline__ void vcombine_state(const SmParams &p, int G, float (&m)[4], float (&d)[4]) {
    if constexpr (VH == 1) {
        merge<kScores>(m[0], d[0], m[1], d[1]);
        merge<kScores>(m[2], d[2], m[3], d[3]);
        merge<kScores>(m[0], d[0], m[2], d[2]);
        m[1] = m[2] = m[3] = m[0];
        d[1] = d[2] = d[3] = d[0];
    } else if constexpr (VH == 2) {
        merge<kScores>(m[0], d[0], m[2], d[2]);
        merge<kScores>(m[1], d[1], m[3], d[3]);
        m[2] = m[0], d[2] = d[0], m[3] = m[1], d[3] = d[1];
    }
    for (int off = VH == 4 ? static_cast<int>(p.H >> 2) : 1; off < G; off <<= 1)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float m2 = __shfl_xor(m[i], off, kWave);
            const float d2 = __shfl_xor(d[i], off, kWave);
            merge<kScores>(m[i], d[i], m2, d2);
        }
}

template <int SRC, int VH>
__device__ __forceinline__ void row_adst(const SmParams &p, int64_t r, int l, float (&adst)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) adst[i] = 0.f;
    if constexpr (SRC == kGat) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t h = VH == 4 ? ((4 * (int64_t)l) & (p.H - 1)) + i : (i & (p.H - 1));
            adst[i] = p.a_dst[r * p.H + h];
        }
    }
}

// State of the flat range [lo, hi) of row r over a group of G lanes, one
// online pass in batches of R blocks per lane: forward (m, d) per element
// position, backward (t, -) with t = sum alpha * g.
template <int SRC, int R, int VH>
__device__ __forceinline__ void vstate(const SmParams &p, int64_t r, int64_t lo, int64_t hi, int G, int l,
                                       float (&m)[4], float (&d)[4]) {
    float adst[4];
    row_adst<SRC, VH>(p, r, l, adst);
    const int64_t b0 = lo >> 2, b1 = (hi + 3) >> 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m[i] = SRC == kBackward ? 0.f : -INFINITY;
        d[i] = 0.f;
    }
    for (int64_t base = b0; base < b1; base += (int64_t)G * R) {
        float v[R][4], gv[R][4];
#pragma unroll
        for (int k = 0; k < R; ++k) {
            const int64_t b = base + l + (int64_t)G * k;
            if (b < b1) {
                vload<SRC, VH>(p, b, lo, hi, adst, v[k], gv[k]);
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) v[k][i] = pad_value<SRC>(), gv[k][i] = 0.f;
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (SRC == kBackward) {
#pragma unroll
                for (int k = 0; k < R; ++k) m[i] = fmaf(v[k][i], gv[k][i], m[i]);
            } else {
                float bm = v[0][i];
#pragma unroll
                for (int k = 1; k < R; ++k) bm = fmaxf(bm, v[k][i]);
                const float mn = fmaxf(m[i], bm);
                if (mn != -INFINITY) {
                    float acc = pexp(m[i], mn) * d[i];
#pragma unroll
                    for (int k = 0; k < R; ++k) acc += pexp(v[k][i], mn);
                    d[i] = acc;
                    m[i] = mn;
                }
            }
        }
    }
    if constexpr (SRC == kBackward) vcombine<VH>(p, G, m, [](float a, float b) { return a + b; });
    else vcombine_state<VH>(p, G, m, d);
}

// Outputs of the flat range [lo, hi) of row r from the row's state.
template <int SRC, int R, int VH>
__device__ __forceinline__ void vwrite(const SmParams &p, int64_t r, int64_t lo, int64_t hi, int G, int l,
                                       const float (&m)[4], const float (&d)[4]) {
    float adst[4], inv[4];
    row_adst<SRC, VH>(p, r, l, adst);
#pragma unroll
    for (int i = 0; i < 4; ++i) inv[i] = SRC == kBackward ? 0.f : 1.f / d[i];
    const int64_t b0 = lo >> 2, b1 = (hi + 3) >> 2;
    for (int64_t base = b0; base < b1; base += (int64_t)G * R) {
        float v[R][4], gv[R][4];
#pragma unroll
        for (int k = 0; k < R; ++k) {
            const int64_t b = base + l + (int64_t)G * k;
            if (b < b1) vload<SRC, VH>(p, b, lo, hi, adst, v[k], gv[k]);
        }
#pragma unroll
        for (int k = 0; k < R; ++k) {
            const int64_t b = base + l + (int64_t)G * k;
            if (b >= b1) continue;
            float o[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                o[i] = SRC == kBackward ? v[k][i] * (gv[k][i] - m[i]) : pexp(v[k][i], m[i]) * inv[i];
            vstore<VH>(p, b, lo, hi, o);
        }
    }
}

// A whole row: read once when it fits R blocks per lane of the group.
template <int SRC, int R, int VH>
__device__ __forceinline__ void vrow(const SmParams &p, int64_t r, int64_t s, int64_t t, int G, int l) {
    const int64_t lo = s * p.H, hi = t * p.H;
    const int64_t b0 = lo >> 2, b1 = (hi + 3) >> 2;
    float m[4], d[4];
    if (b1 - b0 > (int64_t)G * R) {  // too large for registers: online pass, then a second read
        vstate<SRC, PYG_SOFTMAX_STREAM, VH>(p, r, lo, hi, G, l, m, d);
        vwrite<SRC, PYG_SOFTMAX_STREAM, VH>(p, r, lo, hi, G, l, m, d);
        return;
    }
    float adst[4];
    row_adst<SRC, VH>(p, r, l, adst);
    const int K = static_cast<int>((b1 - b0 + G - 1) / G);  // blocks per lane, the same in the whole group
    float v[R][4], gv[R][4];
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const int64_t b = b0 + l + (int64_t)G * k;
        if (b < b1) {
            vload<SRC, VH>(p, b, lo, hi, adst, v[k], gv[k]);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) v[k][i] = pad_value<SRC>(), gv[k][i] = 0.f;
        }
    }
    if constexpr (SRC == kBackward) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            m[i] = 0.f;
#pragma unroll
            for (int k = 0; k < R; ++k)
                if (k < K) m[i] = fmaf(v[k][i], gv[k][i], m[i]);
        }
        vcombine<VH>(p, G, m, [](float a, float b) { return a + b; });
#pragma unroll
        for (int k = 0; k < R; ++k)
            if (k < K)
#pragma unroll
                for (int i = 0; i < 4; ++i) v[k][i] = v[k][i] * (gv[k][i] - m[i]);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            m[i] = v[0][i];
#pragma unroll
            for (int k = 1; k < R; ++k)
                if (k < K) m[i] = fmaxf(m[i], v[k][i]);
        }
        vcombine<VH>(p, G, m, [](float a, float b) { return fmaxf(a, b); });
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            d[i] = 0.f;
#pragma unroll
            for (int k = 0; k < R; ++k)
                if (k < K) {
                    v[k][i] = pexp(v[k][i], m[i]);
                    d[i] += v[k][i];
                }
        }
        vcombine<VH>(p, G, d, [](float a, float b) { return a + b; });
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float inv = 1.f / d[i];
#pragma unroll
            for (int k = 0; k < R; ++k)
                if (k < K) v[k][i] *= inv;
        }
    }
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const int64_t b = b0 + l + (int64_t)G * k;
        if (b < b1) vstore<VH>(p, b, lo, hi, v[k]);
    }
}

// Piece state of a long row over the whole wavefront, stored per head.
template <int SRC, int R, int VH>
__device__ __forceinline__ void vpiece_state(const SmParams &p, int64_t r, int64_t s, int64_t t, int64_t slot,
                                             int lane) {
    float m[4], d[4];
    vstate<SRC, R, VH>(p, r, s * p.H, t * p.H, kWave, lane, m, d);
    const int64_t nl = VH == 4 ? (p.H >> 2) : 1;  // lanes 0 .. nl-1 hold every head once
    if (lane < nl) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t h = VH == 4 ? 4 * (int64_t)lane + i : i;
            if (h < p.H) p.part[slot * p.H + h] = make_float2(m[i], d[i]);
        }
    }
}

template <int SRC, int VH>
__device__ __forceinline__ void do_row(const SmParams &p, int64_t r, int64_t s, int64_t t, int lg_g, int l) {
    if constexpr (VH > 0) {
        vrow<SRC, SRC == kBackward ? PYG_SOFTMAX_REGS_BWD : PYG_SOFTMAX_REGS, VH>(p, r, s, t, 1 << lg_g, l);
    } else {
        for (int64_t hb = 0; hb < p.H; hb += (1 << p.lg_h)) {
            const float2 st = row_state<SRC>(p, r, s, t, hb, lg_g, l);
            row_write<SRC>(p, r, s, t, hb, lg_g, l, st);
        }
    }
}

template <int SRC, int VH>
__device__ __forceinline__ void do_piece(const SmParams &p, int64_t r, int64_t s, int64_t t, int64_t slot, int lane) {
    if constexpr (VH > 0) vpiece_state<SRC, PYG_SOFTMAX_STREAM, VH>(p, r, s, t, slot, lane);
    else piece_state<SRC>(p, r, s, t, slot, lane);
}

// VH: 0 = scalar path; 1, 2 = vector path with H = 1, 2; 4 = vector path with H >= 4.
template <int SRC, int VH>
__global__ __launch_bounds__(kBlock) void k_softmax(SmParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave));
    if (c >= p.nchunks) return;
    const int64_t e0 = c * p.chunk;
    const int64_t e1 = (e0 + p.chunk) < p.E ? (e0 + p.chunk) : p.E;
    const int64_t rA = uniform64(wave_lower_bound(p.rowptr, p.n_rows + 1, e0, lane));
    const int64_t rpA = uniform64(p.rowptr[rA]);
    int32_t cont = -1, head = -1;

    // a long row that started in an earlier chunk: its piece in this chunk
    if (rA > 0 && rpA > e0) {
        const int64_t s0 = uniform64(p.rowptr[rA - 1]);
        if (rpA - s0 > p.chunk) {
            do_piece<SRC, VH>(p, rA - 1, e0, rpA < e1 ? rpA : e1, 2 * c, lane);
            cont = static_cast<int32_t>(rA - 1);
        }
    }
    // rows whose first slot lies in [e0, e1): groups of G lanes take one row each
    const int lg_g = p.lg_g;
    const int S = kWave >> lg_g;
    const int sg = lane >> lg_g;
    const int l = lane & ((1 << lg_g) - 1);
    int64_t rb = rA;
    while (rb < p.n_rows) {
        const int64_t rp = p.rowptr[(rb + lane) < p.n_rows ? (rb + lane) : p.n_rows];
        // lanes 0 .. cnt-1 hold the starts of rows rb .. rb+cnt-1; lane i+1 the end of row rb+i
        const bool in = lane < kWave - 1 && rb + lane < p.n_rows && rp < e1;
        const int cnt = __popcll(__ballot(in));
        const int64_t s_first = lane_value64(rp, 0);
        if (cnt == kWave - 1 && lane_value64(rp, kWave - 1) == s_first) {
            // 63 empty rows in a row (no slots, no output): go on at the last row that starts at s_first
            rb = uniform_lower_bound(p.rowptr, p.n_rows + 1, s_first + 1) - 1;
            continue;
        }
        for (int i0 = 0; i0 < cnt; i0 += S) {
            const int i = i0 + sg;
            const int ii = i < cnt ? i : cnt - 1;
            const int64_t s = __shfl(rp, ii, kWave), t = __shfl(rp, ii + 1, kWave);
            const bool is_long = i < cnt && t - s > p.chunk;  // only the chunk's last row can be long
            const uint64_t lm = __ballot(is_long);
            if (lm) head = static_cast<int32_t>(rb + i0 + ((__ffsll(static_cast<unsigned long long>(lm)) - 1) >> lg_g));
            if (i < cnt && !is_long && t > s) do_row<SRC, VH>(p, rb + i, s, t, lg_g, l);  // uniform within the group
        }
        if (cnt < kWave - 1) break;  // the chunk's rows end in this batch
        rb += cnt;
    }
    head = __builtin_amdgcn_readfirstlane(head);
    if (head >= 0) do_piece<SRC, VH>(p, head, uniform64(p.rowptr[head]), e1, 2 * c + 1, lane);
    if (lane == 0) {
        p.head_row[c] = head;
        p.cont_row[c] = cont;
    }
}

// Fold the piece states of the long row that starts in chunk c, in chunk order.
template <int SRC>
__global__ __launch_bounds__(kBlock) void k_softmax_fold(SmParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave));
    if (c >= p.nchunks) return;
    const int32_t r = p.head_row[c];
    if (r < 0) return;
    const int64_t t = p.rowptr[r + 1];
    const int64_t K = (t - 1) / p.chunk - c + 1;  // pieces of this row
    for (int64_t h = lane; h < p.H; h += kWave) {
        float2 st = identity_state<SRC>();
        for (int64_t mm = 0; mm < K; ++mm) {
            const int64_t slot = mm == 0 ? 2 * c + 1 : 2 * (c + mm);
            const float2 o = p.part[slot * p.H + h];
            merge<SRC>(st.x, st.y, o.x, o.y);
        }
        p.stat[c * p.H + h] = st;
    }
}

// Normalise the long-row pieces of chunk c with their rows' folded states.
template <int SRC, int VH>
__global__ __launch_bounds__(kBlock) void k_softmax_long(SmParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave));
    if (c >= p.nchunks) return;
    const int64_t e0 = c * p.chunk;
    const int64_t e1 = (e0 + p.chunk) < p.E ? (e0 + p.chunk) : p.E;
    const int32_t rows[2] = {p.cont_row[c], p.head_row[c]};
    for (int k = 0; k < 2; ++k) {
        const int64_t r = rows[k];
        if (r < 0) continue;
        const int64_t rs = uniform64(p.rowptr[r]), rt = uniform64(p.rowptr[r + 1]);
        const int64_t s = k == 0 ? e0 : rs;
        const int64_t t = k == 0 ? (rt < e1 ? rt : e1) : e1;
        const int64_t hc = k == 0 ? rs / p.chunk : c;  // chunk that owns the row's folded state
        if constexpr (VH > 0) {
            float m[4], d[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t h = VH == 4 ? ((4 * (int64_t)lane) & (p.H - 1)) + i : (i & (p.H - 1));
                const float2 st = p.stat[hc * p.H + h];
                m[i] = st.x;
                d[i] = st.y;
            }
            vwrite<SRC, PYG_SOFTMAX_STREAM, VH>(p, r, s * p.H, t * p.H, kWave, lane, m, d);
            continue;
        }
        for (int64_t hb = 0; hb < p.H; hb += (1 << p.lg_h)) {
            const int64_t h = hb + (lane & ((1 << p.lg_h) - 1));
            const float2 st = h < p.H ? p.stat[hc * p.H + h] : identity_state<SRC>();
            row_write<SRC>(p, r, s, t, hb, 6, lane, st);
        }
    }
}

struct SmWs {
    float2 *part;
    float2 *stat;
    int32_t *head_row;
    int32_t *cont_row;
    size_t bytes;
};

// Default chunk of the softmax: the segment kernel's, but long-row graphs
// keep 2048 slots per wavefront (1024 or 512 measured slower here, e.g. the
// scores-given softmax 1.95 -> 2.09 ms at 512 on the large power-law graph).
int64_t softmax_chunk(int64_t E, int64_t n_rows, int64_t requested) {
    if (requested > 0 || (n_rows > 0 && E <= 16 * n_rows)) return segment_chunk(E, n_rows, requested);
    int64_t c = 64;
    while (c < 2048 && c * 32768 < E) c <<= 1;
    return c;
}

SmWs carve_softmax(void *base, int64_t E, int64_t H, int64_t chunk) {
    const int64_t nchunks = E > 0 ? (E + chunk - 1) / chunk : 0;
    Carver c(base);
    SmWs w{};
    w.part = c.take<float2>(2 * nchunks * H);
    w.stat = c.take<float2>(nchunks * H);
    w.head_row = c.take<int32_t>(nchunks);
    w.cont_row = c.take<int32_t>(nchunks);
    w.bytes = c.used + 256;
    return w;
}

int ceil_log2(int64_t v) {
    int k = 0;
    while ((int64_t(1) << k) < v && k < 62) ++k;
    return k;
}

template <int SRC>
int run_softmax(SmParams p, const pyg_csr *csr, void *ws, size_t ws_bytes, hipStream_t s) {
    if (p.E == 0 || p.H == 0) return PYG_OK;
    p.chunk = softmax_chunk(p.E, p.n_rows, csr->chunk);
    p.nchunks = (p.E + p.chunk - 1) / p.chunk;
    const SmWs w = carve_softmax(ws, p.E, p.H, p.chunk);
    if (!ws || ws_bytes < w.bytes) return PYG_ERR_WORKSPACE;
    p.part = w.part;
    p.stat = w.stat;
    p.head_row = w.head_row;
    p.cont_row = w.cont_row;
    p.lg_h = ceil_log2(p.H) < 6 ? ceil_log2(p.H) : 6;
    p.lg_hh = ceil_log2(p.H);
    const int64_t avg = (p.E + p.n_rows - 1) / p.n_rows;
    auto al16 = [](const void *q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    // vector path: H a power of two with at most 64 lanes per slot, 16-byte aligned arrays
    const bool vec = (p.H & (p.H - 1)) == 0 && p.H <= 256 && al16(p.out) && al16(p.s) && al16(p.g) &&
                     (SRC != kGat || p.H < 4 || al16(p.a_src));
    int lg;
    if (vec) {  // lanes per short row: about one 16-byte block per lane, at least H/4
        const int lg_min = p.H >= 4 ? p.lg_hh - 2 : 0;
        lg = ceil_log2((avg * p.H + 3) / 4);
        lg = lg < lg_min ? lg_min : lg;
    } else {    // about one lane per element of the mean row, at least Hq
        lg = p.lg_h + ceil_log2(avg);
    }
    p.lg_g = lg < 6 ? lg : 6;
    const unsigned grid = static_cast<unsigned>((p.nchunks + (kBlock / kWave) - 1) / (kBlock / kWave));
    const int vh = !vec ? 0 : (p.H >= 4 ? 4 : static_cast<int>(p.H));
    if (vh == 4) k_softmax<SRC, 4><<<grid, kBlock, 0, s>>>(p);
    else if (vh == 2) k_softmax<SRC, 2><<<grid, kBlock, 0, s>>>(p);
    else if (vh == 1) k_softmax<SRC, 1><<<grid, kBlock, 0, s>>>(p);
    else k_softmax<SRC, 0><<<grid, kBlock, 0, s>>>(p);
    PYG_LAUNCH_CHECK();
    if (p.nchunks > 1) {
        k_softmax_fold<SRC><<<grid, kBlock, 0, s>>>(p);
        PYG_LAUNCH_CHECK();
        if (vh == 4) k_softmax_long<SRC, 4><<<grid, kBlock, 0, s>>>(p);
        else if (vh == 2) k_softmax_long<SRC, 2><<<grid, kBlock, 0, s>>>(p);
        else if (vh == 1) k_softmax_long<SRC, 1><<<grid, kBlock, 0, s>>>(p);
        else k_softmax_long<SRC, 0><<<grid, kBlock, 0, s>>>(p);
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}

int check_csr(const pyg_csr *csr, int order) {
    if (!csr || csr->N < 0 || csr->E < 0) return PYG_ERR_INVALID_ARG;
    if (csr->E > 0 && (!csr->rowptr || !csr->col)) return PYG_ERR_INVALID_ARG;
    if (csr->N > 0 && !csr->rowptr) return PYG_ERR_INVALID_ARG;
    if (csr->E > 0 && csr->N == 0) return PYG_ERR_INVALID_ARG;
    if (csr->E >= (int64_t(1) << 31) || csr->N >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (order != PYG_ORDER_CSR && order != PYG_ORDER_COO) return PYG_ERR_INVALID_ARG;
    if (order == PYG_ORDER_COO && csr->E > 0 && !csr->perm) return PYG_ERR_INVALID_ARG;
    return PYG_OK;
}

SmParams base_params(const pyg_csr *csr, int64_t H, int order, float *out) {
    SmParams p{};
    p.rowptr = csr->rowptr;
    p.col = csr->col;
    p.perm = order == PYG_ORDER_COO ? csr->perm : nullptr;
    p.n_rows = csr->N;
    p.E = csr->E;
    p.H = H;
    p.out = out;
    return p;
}

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" int pyg_segment_softmax_workspace(int64_t E, int64_t N, int64_t H, int64_t chunk, size_t *bytes) {
    if (!bytes || E < 0 || N < 0 || H < 0 || chunk < 0) return PYG_ERR_INVALID_ARG;
    *bytes = E > 0 ? carve_softmax(nullptr, E, H, softmax_chunk(E, N, chunk)).bytes : 0;
    return PYG_OK;
}

extern "C" int pyg_segment_softmax(const float *scores, int64_t H, const pyg_csr *csr, int order, float *alpha,
                                   void *ws, size_t ws_bytes, void *stream) {
    PYG_TRY(check_csr(csr, order));
    if (H <= 0) return PYG_ERR_INVALID_ARG;
    if (csr->E > 0 && (!scores || !alpha)) return PYG_ERR_INVALID_ARG;
    SmParams p = base_params(csr, H, order, alpha);
    p.s = scores;
    return run_softmax<kScores>(p, csr, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

extern "C" int pyg_gat_softmax(const float *a_src, const float *a_dst, int64_t H, float negative_slope,
                               const pyg_csr *csr, int order, float *alpha, void *ws, size_t ws_bytes, void *stream) {
    PYG_TRY(check_csr(csr, order));
    if (H <= 0 || !isfinite(negative_slope)) return PYG_ERR_INVALID_ARG;
    if (csr->E > 0 && (!a_src || !a_dst || !alpha)) return PYG_ERR_INVALID_ARG;
    SmParams p = base_params(csr, H, order, alpha);
    p.a_src = a_src;
    p.a_dst = a_dst;
    p.slope = negative_slope;
    return run_softmax<kGat>(p, csr, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

extern "C" int pyg_segment_softmax_backward(const float *alpha, const float *grad_alpha, int64_t H, const pyg_csr *csr,
                                            int order, float *grad_scores, void *ws, size_t ws_bytes, void *stream) {
    PYG_TRY(check_csr(csr, order));
    if (H <= 0) return PYG_ERR_INVALID_ARG;
    if (csr->E > 0 && (!alpha || !grad_alpha || !grad_scores)) return PYG_ERR_INVALID_ARG;
    SmParams p = base_params(csr, H, order, grad_scores);
    p.s = alpha;
    p.g = grad_alpha;
    return run_softmax<kBackward>(p, csr, ws, ws_bytes, static_cast<hipStream_t>(stream));
}
