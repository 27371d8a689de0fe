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
// holding its first slot and is done there in two passes over its slots:
// an online max/sum pass (one exp per element, rescaling when the running
// maximum grows) and a normalising pass. Lanes are split into groups of G
// lanes per row; inside a group Hq lanes (H rounded up to a power of two,
// at most 64) cover the heads of one slot and G / Hq slots go side by side,
// so consecutive lanes read consecutive addresses. Short rows share a
// wavefront (G < 64) when the mean degree is small.
// A longer row is cut at chunk boundaries: every piece's (max, sum) goes to
// a partial, a fold kernel merges the partials of each long row in chunk
// order, and a third kernel normalises the pieces. All orders are fixed, so
// results are bit-reproducible.
#include "common.hpp"

#include <math.h>

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
    int lg_h;  // log2 of lanes per slot (Hq)
    int lg_g;  // log2 of lanes per short row
    float *out;
    float2 *part;       // [2 * nchunks, H]: piece states (continuing piece at 2c, head piece at 2c + 1)
    float2 *stat;       // [nchunks, H]: folded state of the long row that starts in chunk c
    int32_t *head_row;  // [nchunks]: long row starting in chunk c, or -1
    int32_t *cont_row;  // [nchunks]: long row continuing into chunk c, or -1
};

// Running state of one (row, head): forward (m = max, d = sum exp(v - m)),
// backward (m = sum alpha * g, d unused).
template <int SRC>
__device__ __forceinline__ void merge(float &m, float &d, float m2, float d2) {
    if constexpr (SRC == kBackward) {
        m += m2;
    } else {
        if (m2 > m) {
            d = d * expf(m - m2) + d2;
            m = m2;
        } else if (m2 != -INFINITY) {
            d += d2 * expf(m2 - m);
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
        d = d * expf(m - v) + 1.f;
        m = v;
    } else {
        d += expf(v - m);
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
            else p.out[e[u]] = expf(v[u] - st.x) * inv;
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

template <int SRC>
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
            piece_state<SRC>(p, rA - 1, e0, rpA < e1 ? rpA : e1, 2 * c, lane);
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
        for (int i0 = 0; i0 < cnt; i0 += S) {
            const int i = i0 + sg;
            const int ii = i < cnt ? i : cnt - 1;
            const int64_t s = __shfl(rp, ii, kWave), t = __shfl(rp, ii + 1, kWave);
            const bool is_long = i < cnt && t - s > p.chunk;  // only the chunk's last row can be long
            const uint64_t lm = __ballot(is_long);
            if (lm) head = static_cast<int32_t>(rb + i0 + ((__ffsll(static_cast<unsigned long long>(lm)) - 1) >> lg_g));
            if (i < cnt && !is_long && t > s) {  // uniform within the group
                for (int64_t hb = 0; hb < p.H; hb += (1 << p.lg_h)) {
                    const float2 st = row_state<SRC>(p, rb + i, s, t, hb, lg_g, l);
                    row_write<SRC>(p, rb + i, s, t, hb, lg_g, l, st);
                }
            }
        }
        if (cnt < kWave - 1) break;  // the chunk's rows end in this batch
        rb += cnt;
    }
    head = __builtin_amdgcn_readfirstlane(head);
    if (head >= 0) piece_state<SRC>(p, head, uniform64(p.rowptr[head]), e1, 2 * c + 1, lane);
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
template <int SRC>
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
    p.chunk = segment_chunk(p.E, p.n_rows, csr->chunk);
    p.nchunks = (p.E + p.chunk - 1) / p.chunk;
    const SmWs w = carve_softmax(ws, p.E, p.H, p.chunk);
    if (!ws || ws_bytes < w.bytes) return PYG_ERR_WORKSPACE;
    p.part = w.part;
    p.stat = w.stat;
    p.head_row = w.head_row;
    p.cont_row = w.cont_row;
    p.lg_h = ceil_log2(p.H) < 6 ? ceil_log2(p.H) : 6;
    // lanes per short row: about one lane per element of the mean row, at least Hq
    const int64_t avg = (p.E + p.n_rows - 1) / p.n_rows;
    const int lg = p.lg_h + ceil_log2(avg);
    p.lg_g = lg < 6 ? lg : 6;
    const unsigned grid = static_cast<unsigned>((p.nchunks + (kBlock / kWave) - 1) / (kBlock / kWave));
    k_softmax<SRC><<<grid, kBlock, 0, s>>>(p);
    PYG_LAUNCH_CHECK();
    if (p.nchunks > 1) {
        k_softmax_fold<SRC><<<grid, kBlock, 0, s>>>(p);
        PYG_LAUNCH_CHECK();
        k_softmax_long<SRC><<<grid, kBlock, 0, s>>>(p);
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
    *bytes = E > 0 ? carve_softmax(nullptr, E, H, segment_chunk(E, N, chunk)).bytes : 0;
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
