// Target-sorted (CSR) segment reduction on gfx950: the propagate kernel
// that reads a row-ordered edge list, and the same machinery for global
// pooling (rows = graphs, slots = nodes).
//
// Work split: the E CSR slots are cut into equal chunks of `chunk` slots and
// each 64-lane wavefront owns one chunk, so every wavefront gathers the same
// number of source rows whatever the degree skew. A row whose degree is at
// most `chunk` is reduced entirely by the wavefront whose chunk holds its
// first slot (it may run past the chunk end). A longer row is cut at chunk
// boundaries; each wavefront writes its piece as a partial and a second
// kernel folds the pieces in chunk order. Every reduction order is fixed, so
// results are bit-reproducible.
//
// Inside a wavefront: L lanes cover one feature row (16-byte vectors when
// rows are 16-byte aligned), S = 64 / L sub-groups take successive edges of
// the row, each lane keeps U gathers in flight, and the sub-groups are
// combined with a butterfly of cross-lane shuffles. Column indices and
// weights are read once per 64 edges, coalesced, and handed to sub-groups
// through ds_bpermute. There is no matrix-core work: aggregation is not a
// dense contraction.
//
// Cache hint for the row gathers: in a power-law graph a few thousand hub
// rows receive a large share of all references (the top 16k of 233k rows
// take half of them), but a stream of one-off rows evicts them from the
// 4 MB L2 of each XCD. When x is larger than L2, a pre-pass histograms the
// rows' degrees in 8 classes per octave and picks the smallest class whose
// rows still fit a 12 MB budget; rows of lower classes are then gathered
// with non-temporal loads, so the hub rows stay cached. Row in-degree stands
// in for how often a row is read as a source (equal on undirected graphs);
// the hint changes only the cache policy, never the result.
//
// Narrow windows: for large inputs with rows wider than a cache line, the
// plain messages run over 128-byte feature windows (one line gathered per
// slot, 8 lanes per sub-group), all windows in one launch, window-major, and
// long rows are folded once after it; the hint is then off. Each window's reduction order
// is fixed, so results stay bit-reproducible.
#include "common.hpp"

#include <type_traits>

#ifndef PYG_SEG_MAX_CHUNK
#define PYG_SEG_MAX_CHUNK 1024  // default chunk of long-row graphs (slots per wavefront), at most
#endif
#ifndef PYG_MIN_CHUNKS
#define PYG_MIN_CHUNKS 4096  // chunk halved (down to 16 slots) while there are fewer chunks than this
#endif

namespace pyg {
namespace {

struct SegParams {
    const void *x;
    int64_t F;      // row stride of x, out and partials (elements)
    int64_t fbase;  // first feature of this launch's window
    int64_t fcnt;   // features in the window
    int64_t nwin;   // > 1: this launch covers nwin windows of fcnt features, window-major
    const int64_t *rowptr;
    const int32_t *col;
    const float *w;
    const float *alpha;  // per-head weights [E, H] in slot order (kMsgHeads)
    const int32_t *alpha_idx;  // non-NULL: slot p takes row alpha_idx[p] of alpha
    const void *ea;           // edge features [E, F] in x's dtype (edge messages)
    const int64_t *ea_perm;   // non-NULL: ea is in COO order, row perm[slot]
    const int32_t *ea_idx;    // non-NULL: ea row ea_idx[slot] (takes precedence over ea_perm)
    const void *x_self;       // kMsgEdgeReluGrad: the rows' own x [n_rows, F]
    int64_t H;
    int64_t C;           // columns per head: feature f belongs to head f / C
    const int64_t *perm;
    int64_t n_rows;
    int64_t E;
    int64_t chunk;
    int64_t nchunks;
    int lg_l;  // log2 of lanes per feature row
    int mean;
    int64_t sentinel;
    void *out;
    int64_t *argmax;
    float *part_val;
    int32_t *part_pos;
    int32_t *head_row;
    const int32_t *hot_class;  // rows of degree class below *hot_class are gathered non-temporally; NULL = no hint
    int32_t *class_hist;       // workspace for the hint pre-pass
    int32_t *hot_slot;
    uint8_t *node_class;       // degree class of every row [n_rows]
    // source-blocked rows: the rows are `blocks` runs of `rpb` virtual rows,
    // virtual row r = (source block r / rpb, target r % rpb)
    int64_t blocks;
    int64_t rpb;
    // > 0: the launch's first zero_items work items zero-fill every empty row
    // (all F features), zero_rows rows each; the row walkers skip long runs
    // of empty rows, so one launch of every call must carry them
    int64_t zero_items;
    int64_t zero_rows;  // rows per zero-fill work item (a multiple of 64)
    // GCN messages (kMsgGcn): dinv [n_rows] fp64 (d^-1/2 of every row), the
    // slot weight w_p = dinv[col] * w_p * dinv[row] formed in fp64 and rounded
    // once; norm_out [E] (or NULL) receives it from the window at feature 0
    const double *dinv;
    float *norm_out;
};

// Measured on the large power-law graph (F = 128): fp32 rows (512 B) gain
// 10 % with a 8-12 MB hot budget; bf16 rows (256 B) lose at every budget, so
// the hint is used for rows of at least 512 B only.
#ifndef PYG_LIGHT_MAX_DEGREE
#define PYG_LIGHT_MAX_DEGREE 16  // kNN rows of 16 slots gain 25 % as light rows
#endif
constexpr int64_t kLightMaxDegree = PYG_LIGHT_MAX_DEGREE;  // mean row length up to which rows go to sub-groups
// Source arrays from 64 MB: the 39 MB PubMed-shaped rows (F = 500) lose 20 %
// with the hint, the 119 MB large-graph rows gain 10 %.
#ifndef PYG_HINT_MIN_MB
#define PYG_HINT_MIN_MB 64
#endif
constexpr int64_t kHintMinBytes = (int64_t)PYG_HINT_MIN_MB << 20;
constexpr int64_t kHintMinRowBytes = 512;
constexpr int64_t kHotBudgetBytes = 12ll << 20;  // hot rows kept cacheable
// Narrow windows: when the source rows are large in total and wider than one
// cache line, the row is reduced one 128-byte window (32 fp32 / 64 bf16
// features) at a time. Every wavefront then gathers a single line per slot,
// a sub-group needs only 8 lanes (8 slots in flight per wavefront instead of
// 2 for 512-byte rows), and the wavefronts in flight work on one window at a
// time (the launch is window-major), so the lines they reuse are a quarter
// of the rows' bytes and far more of them stay in L2. The index stream is
// read once per window (8 B per slot). One launch for all windows instead of
// one per window leaves a single drain tail: 5.44 -> 5.35 ms. Measured on
// the large power-law graph (F = 128): fp32 6.52 -> 5.43 ms, bf16 3.12 ->
// 2.69 ms; 256-byte windows 6.77 ms. Graphs whose rows total under 16 MB
// lose (more launches for rows that fit in L2 anyway), so they keep whole
// rows. Only the plain messages: per-head weights and edge features are read
// again by every window, and those kinds lose (heads backward 16.4 -> 22.7
// ms, bf16 edge features 8.7 -> 9.5 ms). The cache hint is off with narrow
// windows (on, at any budget, 5.4 -> 8.2 ms and more).
#ifndef PYG_WINDOW_BYTES
#define PYG_WINDOW_BYTES 128
#endif
#ifndef PYG_WINDOW_MIN_MB
#define PYG_WINDOW_MIN_MB 16
#endif
#ifndef PYG_NARROW_ALL
#define PYG_NARROW_ALL 0  // 1: narrow windows for every message kind
#endif
#ifndef PYG_WINDOWS_ONE_LAUNCH
#define PYG_WINDOWS_ONE_LAUNCH 1  // 0: one launch per narrow window
#endif
#ifndef PYG_HINT_NARROW
#define PYG_HINT_NARROW 0  // 0: no hint with narrow windows; 1: hot budget counted in window bytes; 2: in row bytes
#endif
constexpr int64_t kWindowBytes = PYG_WINDOW_BYTES;
constexpr int64_t kWindowMinBytes = (int64_t)PYG_WINDOW_MIN_MB << 20;

// ------------------------------------------------------- lane vector types
template <typename T, bool VEC> struct Lane;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <> struct Lane<float, true> {  // 4 x fp32 = 16 B
    using R = float4;
    static constexpr int N = 4;
    __device__ static R load(const float *p) { return *reinterpret_cast<const R *>(p); }
    __device__ static R load_nt(const float *p) {
        const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(p));
        return make_float4(v.x, v.y, v.z, v.w);
    }
    __device__ static R zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
    __device__ static float get(const R &r, int e) { return e == 0 ? r.x : e == 1 ? r.y : e == 2 ? r.z : r.w; }
    __device__ static void store(float *p, const float (&v)[N]) { *reinterpret_cast<R *>(p) = make_float4(v[0], v[1], v[2], v[3]); }
};
template <> struct Lane<uint16_t, true> {  // 8 x bf16 = 16 B
    using R = uint4;
    static constexpr int N = 8;
    __device__ static R load(const uint16_t *p) { return *reinterpret_cast<const R *>(p); }
    __device__ static R load_nt(const uint16_t *p) {
        const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
        return make_uint4(v.x, v.y, v.z, v.w);
    }
    __device__ static R zero() { return make_uint4(0, 0, 0, 0); }
    __device__ static float get(const R &r, int e) {
        const uint32_t w = (e >> 1) == 0 ? r.x : (e >> 1) == 1 ? r.y : (e >> 1) == 2 ? r.z : r.w;
        return (e & 1) ? __uint_as_float(w & 0xFFFF0000u) : __uint_as_float(w << 16);
    }
    __device__ static void store(uint16_t *p, const float (&v)[N]) {
        uint32_t o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = uint32_t(f32_to_bf16_rne(v[2 * i])) | (uint32_t(f32_to_bf16_rne(v[2 * i + 1])) << 16);
        *reinterpret_cast<R *>(p) = make_uint4(o[0], o[1], o[2], o[3]);
    }
};
template <> struct Lane<float, false> {
    using R = float;
    static constexpr int N = 1;
    __device__ static R load(const float *p) { return *p; }
    __device__ static R load_nt(const float *p) { return __builtin_nontemporal_load(p); }
    __device__ static R zero() { return 0.f; }
    __device__ static float get(const R &r, int) { return r; }
    __device__ static void store(float *p, const float (&v)[N]) { *p = v[0]; }
};
template <> struct Lane<uint16_t, false> {
    using R = uint16_t;
    static constexpr int N = 1;
    __device__ static R load(const uint16_t *p) { return *p; }
    __device__ static R load_nt(const uint16_t *p) { return __builtin_nontemporal_load(p); }
    __device__ static R zero() { return 0; }
    __device__ static float get(const R &r, int) { return bf16_bits_to_f32(r); }
    __device__ static void store(uint16_t *p, const float (&v)[N]) { *p = f32_to_bf16_rne(v[0]); }
};

// Stores one lane's EP results of a row: in the row dtype T, or as fp32
// (OF32: partial rows of source blocks, folded later).
template <typename T, bool VEC, bool OF32>
__device__ __forceinline__ void store_out(void *out, int64_t idx, const float (&v)[Lane<T, VEC>::N]) {
    constexpr int EP = Lane<T, VEC>::N;
    if constexpr (OF32) {
        float *o = static_cast<float *>(out) + idx;
        if constexpr (VEC) {
#pragma unroll
            for (int k = 0; k < EP / 4; ++k)
                reinterpret_cast<float4 *>(o)[k] = make_float4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]);
        } else {
            o[0] = v[0];
        }
    } else {
        Lane<T, VEC>::store(static_cast<T *>(out) + idx, v);
    }
}

// Degree class: 8 classes per octave, monotone in d, 0 for d <= 0.
__device__ __forceinline__ int deg_class(int64_t d) {
    if (d <= 0) return 0;
    const int oct = 63 - __clzll(static_cast<unsigned long long>(d));
    const int sub = oct >= 3 ? static_cast<int>((d >> (oct - 3)) & 7) : static_cast<int>((d << (3 - oct)) & 7);
    const int c = oct * 8 + sub + 1;
    return c < 255 ? c : 255;
}
constexpr int kClasses = 256;

constexpr int kFull = 0, kPartial = 1;
constexpr int kMsgSrc = 0, kMsgWeighted = 1, kMsgDiff = 2, kMsgHeads = 3;
constexpr int kMsgEdgeAdd = 4, kMsgEdgeRelu = 5, kMsgEdgeMul = 6;  // x_j + e, max(x_j + e, 0), x_j * e
// Backward of max(x_r + e, 0) over the reversed graph: the gathered upstream
// gradient where x_r + e > 0, x_r being the row's own features (x_self).
constexpr int kMsgEdgeReluGrad = 7;
// GCN: the weight of slot p is dinv[col[p]] * w_p * dinv[row] (w_p = 1 without weights)
constexpr int kMsgGcn = 8;
// messages whose slot carries a scalar weight (read or formed)
template <int MSG> constexpr bool kWeightedMsg = MSG == 1 || MSG == 8;

// The target of row r: r itself, or for a source-blocked virtual row the
// target it belongs to.
__device__ __forceinline__ int64_t target_row(const SegParams &p, int64_t r) {
    return p.blocks > 1 ? r % p.rpb : r;
}

// Edge-feature message of one element (formed in fp32, as compared by max).
template <int MSG>
__device__ __forceinline__ float edge_msg(float xv, float ev) {
    if constexpr (MSG == kMsgEdgeAdd) return xv + ev;
    else if constexpr (MSG == kMsgEdgeRelu) return (xv + ev) > 0.f ? (xv + ev) : 0.f;
    else return xv * ev;
}

// Reduce slots [s, t) of row r; write the row (kFull) or a partial (kPartial).
template <typename T, bool VEC, int NS, int U, int MSG, bool MAXA, bool IDENT, bool OF32 = false>
__device__ __forceinline__ void reduce_piece(const SegParams &p, int64_t r, int64_t s, int64_t t, int kind,
                                             int64_t slot, int lane, int hot) {
    using LN = Lane<T, VEC>;
    using R = typename LN::R;
    constexpr int EP = LN::N;
    const T *__restrict__ x = static_cast<const T *>(p.x);
    const int L = 1 << p.lg_l;
    const int S = kWave >> p.lg_l;
    const int q = lane & (L - 1);
    const int sg = lane >> p.lg_l;

    int64_t f0[NS];
    bool act[NS];
#pragma unroll
    for (int sl = 0; sl < NS; ++sl) {
        const int64_t fo = ((int64_t)sl * L + q) * EP;
        act[sl] = fo < p.fcnt && p.fbase + fo < p.F;  // the last window of a row may be narrower
        f0[sl] = p.fbase + fo;
    }
    float acc[NS][EP];
    int32_t pos[NS][EP];
#pragma unroll
    for (int sl = 0; sl < NS; ++sl)
#pragma unroll
        for (int e = 0; e < EP; ++e) {
            acc[sl][e] = 0.f;
            pos[sl][e] = -1;
        }
    R xi[NS];
    if constexpr (MSG == kMsgDiff || MSG == kMsgEdgeReluGrad) {
        const T *xr = MSG == kMsgDiff ? x : static_cast<const T *>(p.x_self);
        const int64_t rr = target_row(p, r);
#pragma unroll
        for (int sl = 0; sl < NS; ++sl) xi[sl] = act[sl] ? LN::load(xr + rr * p.F + f0[sl]) : LN::zero();
    }
    // GCN: the row's own d^-1/2
    double dr = 0.0;
    if constexpr (MSG == kMsgGcn) dr = p.dinv[target_row(p, r)];
    // per-head weights: a lane vector never straddles two heads (C is a multiple of its width)
    int64_t hd[NS];
#pragma unroll
    for (int sl = 0; sl < NS; ++sl) hd[sl] = MSG == kMsgHeads ? f0[sl] / p.C : 0;

    // column indices and weights stream once: read them 64 at a time,
    // non-temporally, one batch ahead of the gathers that use them; bit 31 of
    // a column marks a cold source row (gathered non-temporally)
    auto fetch = [&](int64_t e, int &c, float &w, int &ar) {
        if (IDENT) {
            c = static_cast<int>(e);
        } else {
            c = __builtin_nontemporal_load(p.col + e);
            if constexpr (MSG == kMsgGcn) {
                const double wv = p.w ? static_cast<double>(__builtin_nontemporal_load(p.w + e)) : 1.0;
                w = static_cast<float>(p.dinv[c] * wv * dr);
                if (p.norm_out && p.fbase == 0) p.norm_out[e] = w;  // every slot once, by the first window
            }
            if (hot > 0 && p.node_class[c] < hot) c |= static_cast<int>(0x80000000u);
        }
        if constexpr (MSG == kMsgWeighted) w = __builtin_nontemporal_load(p.w + e);
        if constexpr (MSG == kMsgHeads) ar = p.alpha_idx ? __builtin_nontemporal_load(p.alpha_idx + e) : static_cast<int>(e);
    };
    int nxc = 0, nxa = 0;
    float nxw = 1.f;
    if (s + lane < t) fetch(s + lane, nxc, nxw, nxa);
    for (int64_t base = s; base < t; base += kWave) {
        const int n = static_cast<int>(uniform64((t - base) < kWave ? (t - base) : kWave));
        const int myc = nxc;
        const float myw = nxw;
        const int mya = nxa;
        if (base + kWave + lane < t) fetch(base + kWave + lane, nxc, nxw, nxa);
        for (int st = 0; st < n; st += S * U) {
            int jj[U], aa[U];
            float ww[U];
            bool ok[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = st + u * S + sg;
                ok[u] = idx < n;
                jj[u] = __shfl(myc, idx & (kWave - 1), kWave);
                if constexpr (kWeightedMsg<MSG>) ww[u] = __shfl(myw, idx & (kWave - 1), kWave);
                if constexpr (MSG == kMsgHeads) aa[u] = __shfl(mya, idx & (kWave - 1), kWave);
            }
            float wh[U][NS];
            if constexpr (MSG == kMsgHeads) {
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int sl = 0; sl < NS; ++sl)
                        wh[u][sl] = (ok[u] && act[sl]) ? p.alpha[(int64_t)aa[u] * p.H + hd[sl]] : 0.f;
            }
            constexpr bool EDGE = MSG >= kMsgEdgeAdd;
            R ev[U][NS];
            if constexpr (EDGE) {  // edge rows stream once: non-temporal
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int sl = 0; sl < NS; ++sl) {
                        const int64_t slot = base + st + u * S + sg;
                        ev[u][sl] = LN::zero();
                        if (ok[u] && act[sl]) {
                            const int64_t er = p.ea_idx ? p.ea_idx[slot] : (p.ea_perm ? p.ea_perm[slot] : slot);
                            ev[u][sl] = LN::load_nt(static_cast<const T *>(p.ea) + er * p.F + f0[sl]);
                        }
                    }
            }
            R v[U][NS];
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int sl = 0; sl < NS; ++sl)
                {
                    const T *src = x + (int64_t)(jj[u] & 0x7FFFFFFF) * p.F + f0[sl];
                    if (!(ok[u] && act[sl])) v[u][sl] = LN::zero();
                    else if (jj[u] < 0) v[u][sl] = LN::load_nt(src);
                    else v[u][sl] = LN::load(src);
                }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!ok[u]) continue;
                const int32_t here = static_cast<int32_t>(base + st + u * S + sg);
#pragma unroll
                for (int sl = 0; sl < NS; ++sl)
#pragma unroll
                    for (int e = 0; e < EP; ++e) {
                        const float xv = LN::get(v[u][sl], e);
                        if constexpr (MAXA) {
                            float m;
                            if constexpr (MSG == kMsgDiff) m = xv - LN::get(xi[sl], e);
                            else if constexpr (kWeightedMsg<MSG>) m = ww[u] * xv;
                            else if constexpr (EDGE) m = edge_msg<MSG>(xv, LN::get(ev[u][sl], e));
                            else m = xv;
                            m = canon_zero(m);
                            if (pos[sl][e] < 0 || m > acc[sl][e]) {
                                acc[sl][e] = m;
                                pos[sl][e] = here;
                            }
                        } else {
                            if constexpr (MSG == kMsgDiff) acc[sl][e] += xv - LN::get(xi[sl], e);
                            else if constexpr (kWeightedMsg<MSG>) acc[sl][e] = fmaf(ww[u], xv, acc[sl][e]);
                            else if constexpr (MSG == kMsgHeads) acc[sl][e] = fmaf(wh[u][sl], xv, acc[sl][e]);
                            else if constexpr (MSG == kMsgEdgeMul) acc[sl][e] = fmaf(xv, LN::get(ev[u][sl], e), acc[sl][e]);
                            else if constexpr (MSG == kMsgEdgeReluGrad)
                                acc[sl][e] += LN::get(xi[sl], e) + LN::get(ev[u][sl], e) > 0.f ? xv : 0.f;
                            else if constexpr (EDGE) acc[sl][e] += edge_msg<MSG>(xv, LN::get(ev[u][sl], e));
                            else acc[sl][e] += xv;
                        }
                    }
            }
        }
    }

    // butterfly across sub-groups (fixed order -> deterministic)
    for (int off = L; off < kWave; off <<= 1) {
#pragma unroll
        for (int sl = 0; sl < NS; ++sl)
#pragma unroll
            for (int e = 0; e < EP; ++e) {
                const float o = __shfl_xor(acc[sl][e], off, kWave);
                if constexpr (MAXA) {
                    const int32_t op = __shfl_xor(pos[sl][e], off, kWave);
                    if (op >= 0 && (pos[sl][e] < 0 || o > acc[sl][e] || (o == acc[sl][e] && op < pos[sl][e]))) {
                        acc[sl][e] = o;
                        pos[sl][e] = op;
                    }
                } else {
                    acc[sl][e] += o;
                }
            }
    }
    if (sg != 0) return;

#pragma unroll
    for (int sl = 0; sl < NS; ++sl) {
        if (!act[sl]) continue;
        if (kind == kPartial) {
            float *pv = p.part_val + slot * p.F + f0[sl];
#pragma unroll
            for (int e = 0; e < EP; ++e) pv[e] = acc[sl][e];
            if constexpr (MAXA) {
                int32_t *pp = p.part_pos + slot * p.F + f0[sl];
#pragma unroll
                for (int e = 0; e < EP; ++e) pp[e] = pos[sl][e];
            }
            continue;
        }
        float v[EP];
        const int64_t deg = t - s;
#pragma unroll
        for (int e = 0; e < EP; ++e) {
            if constexpr (MAXA) v[e] = pos[sl][e] >= 0 ? acc[sl][e] : 0.f;
            else v[e] = (p.mean && deg > 0) ? acc[sl][e] / static_cast<float>(deg) : acc[sl][e];
        }
        store_out<T, VEC, OF32>(p.out, r * p.F + f0[sl], v);
        if constexpr (MAXA) {
            int64_t *ap = p.argmax + r * p.F + f0[sl];
#pragma unroll
            for (int e = 0; e < EP; ++e) {
                const int32_t ps = pos[sl][e];
                ap[e] = ps < 0 ? p.sentinel : (p.perm ? p.perm[ps] : static_cast<int64_t>(ps));
            }
        }
    }
}

// Light rows: one sub-group of L lanes reduces a whole short row alone, so a
// wavefront works on S rows at once. `mine` is false for sub-groups without
// a row; nothing below crosses sub-groups, so the branch may diverge.
template <typename T, bool VEC, int U, int MSG, bool MAXA, bool IDENT, bool OF32>
__device__ __forceinline__ void light_row(const SegParams &p, int64_t r, int64_t s, int64_t t, bool mine, int lane) {
    using LN = Lane<T, VEC>;
    using R = typename LN::R;
    constexpr int EP = LN::N;
    if (!mine) return;
    const T *__restrict__ x = static_cast<const T *>(p.x);
    const int q = lane & ((1 << p.lg_l) - 1);
    const int64_t fo = (int64_t)q * EP;
    const bool act = fo < p.fcnt && p.fbase + fo < p.F;  // the last window of a row may be narrower
    const int64_t f0 = p.fbase + fo;
    float acc[EP];
    int32_t pos[EP];
#pragma unroll
    for (int e = 0; e < EP; ++e) {
        acc[e] = 0.f;
        pos[e] = -1;
    }
    R xi = LN::zero();
    const int64_t rr = target_row(p, r);
    if constexpr (MSG == kMsgDiff) xi = act ? LN::load(x + rr * p.F + f0) : LN::zero();
    if constexpr (MSG == kMsgEdgeReluGrad) xi = act ? LN::load(static_cast<const T *>(p.x_self) + rr * p.F + f0) : LN::zero();
    const int64_t hd = MSG == kMsgHeads ? f0 / p.C : 0;
    for (int64_t base = s; base < t; base += U) {
        int jj[U];
        float ww[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {  // every lane of the sub-group reads the same slot
            ok[u] = base + u < t;
            jj[u] = ok[u] ? (IDENT ? static_cast<int>(base + u) : p.col[base + u]) : 0;
            ww[u] = 1.f;
            if constexpr (MSG == kMsgWeighted) ww[u] = ok[u] ? p.w[base + u] : 0.f;
            if constexpr (MSG == kMsgGcn) {
                if (ok[u]) {
                    const double wv = p.w ? static_cast<double>(p.w[base + u]) : 1.0;
                    ww[u] = static_cast<float>(p.dinv[jj[u]] * wv * p.dinv[rr]);
                    if (p.norm_out && p.fbase == 0 && q == 0) p.norm_out[base + u] = ww[u];
                } else {
                    ww[u] = 0.f;
                }
            }
            if constexpr (MSG == kMsgHeads) {
                const int64_t ar = p.alpha_idx ? (ok[u] ? p.alpha_idx[base + u] : 0) : base + u;
                ww[u] = (ok[u] && act) ? p.alpha[ar * p.H + hd] : 0.f;
            }
        }
        constexpr bool EDGE = MSG >= kMsgEdgeAdd;
        R ev[U];
        if constexpr (EDGE) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                ev[u] = LN::zero();
                if (ok[u] && act) {
                    const int64_t er = p.ea_idx ? p.ea_idx[base + u] : (p.ea_perm ? p.ea_perm[base + u] : base + u);
                    ev[u] = LN::load_nt(static_cast<const T *>(p.ea) + er * p.F + f0);
                }
            }
        }
        R v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = (ok[u] && act) ? LN::load(x + (int64_t)jj[u] * p.F + f0) : LN::zero();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (!ok[u]) continue;
#pragma unroll
            for (int e = 0; e < EP; ++e) {
                const float xv = LN::get(v[u], e);
                if constexpr (MAXA) {
                    float m;
                    if constexpr (MSG == kMsgDiff) m = xv - LN::get(xi, e);
                    else if constexpr (kWeightedMsg<MSG>) m = ww[u] * xv;
                    else if constexpr (EDGE) m = edge_msg<MSG>(xv, LN::get(ev[u], e));
                    else m = xv;
                    m = canon_zero(m);
                    if (pos[e] < 0 || m > acc[e]) {
                        acc[e] = m;
                        pos[e] = static_cast<int32_t>(base + u);
                    }
                } else {
                    if constexpr (MSG == kMsgDiff) acc[e] += xv - LN::get(xi, e);
                    else if constexpr (kWeightedMsg<MSG> || MSG == kMsgHeads) acc[e] = fmaf(ww[u], xv, acc[e]);
                    else if constexpr (MSG == kMsgEdgeMul) acc[e] = fmaf(xv, LN::get(ev[u], e), acc[e]);
                    else if constexpr (MSG == kMsgEdgeReluGrad) acc[e] += LN::get(xi, e) + LN::get(ev[u], e) > 0.f ? xv : 0.f;
                    else if constexpr (EDGE) acc[e] += edge_msg<MSG>(xv, LN::get(ev[u], e));
                    else acc[e] += xv;
                }
            }
        }
    }
    if (!act) return;
    float v[EP];
    const int64_t deg = t - s;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
        if constexpr (MAXA) v[e] = pos[e] >= 0 ? acc[e] : 0.f;
        else v[e] = (p.mean && deg > 0) ? acc[e] / static_cast<float>(deg) : acc[e];
    }
    store_out<T, VEC, OF32>(p.out, r * p.F + f0, v);
    if constexpr (MAXA) {
        int64_t *ap = p.argmax + r * p.F + f0;
#pragma unroll
        for (int e = 0; e < EP; ++e) ap[e] = pos[e] < 0 ? p.sentinel : (p.perm ? p.perm[pos[e]] : static_cast<int64_t>(pos[e]));
    }
}

// Empty rows (no slots) are written here, in parallel, rather than by the
// chunk walkers: a run of empty rows all starts at one slot and so belongs to
// one chunk, which would otherwise walk it row by row (a graph whose first
// half of rows has no edges took 70 times longer than one without). Work
// item z covers rows [z * zero_rows, (z + 1) * zero_rows): every empty row
// gets 0 in all F features (and argmax = sentinel). About 1,024 items per
// launch, each a few dependent loads of row bounds.
inline void set_zero_items(SegParams &p, int64_t n_rows) {
    int64_t per = (n_rows + 1023) / 1024;
    per = (per + kWave - 1) / kWave * kWave;
    p.zero_rows = per > kWave ? per : kWave;
    p.zero_items = (n_rows + p.zero_rows - 1) / p.zero_rows;
}
template <typename T, bool OF32>
__device__ __forceinline__ void zero_empty_rows(const SegParams &p, int64_t z, int lane) {
    using TO = typename std::conditional<OF32, float, T>::type;
    TO *out = static_cast<TO *>(p.out);
    const int64_t r_end = (z + 1) * p.zero_rows < p.n_rows ? (z + 1) * p.zero_rows : p.n_rows;
    for (int64_t r0 = z * p.zero_rows; r0 < r_end; r0 += kWave) {
        const int64_t r = r0 + lane;
        const bool in = r < r_end;
        const int64_t a = in ? p.rowptr[r] : 0, b = in ? p.rowptr[r + 1] : 1;
        uint64_t m = __ballot(in && a == b);
        while (m) {
            const int k = __ffsll(static_cast<unsigned long long>(m)) - 1;
            m &= m - 1;
            const int64_t row = r0 + k;
            for (int64_t f = lane; f < p.F; f += kWave) {
                out[row * p.F + f] = TO(0);
                if (p.argmax) p.argmax[row * p.F + f] = p.sentinel;
            }
        }
    }
}

// One wavefront's work on chunk c (features p.fbase .. p.fbase + p.fcnt).
template <typename T, bool VEC, int NS, int U, int MSG, bool MAXA, bool IDENT, bool LIGHT, bool OF32>
__device__ __forceinline__ void segment_chunk_work(const SegParams &p, int64_t c, int lane) {
    const int64_t e0 = c * p.chunk;
    const int64_t e1 = (e0 + p.chunk) < p.E ? (e0 + p.chunk) : p.E;
    const bool last = c == p.nchunks - 1;
    const int64_t rA = uniform64(wave_lower_bound(p.rowptr, p.n_rows + 1, e0, lane));
    const int64_t rpA = uniform64(p.rowptr[rA]);
    const int hot = (!IDENT && p.hot_class) ? __builtin_amdgcn_readfirstlane(*p.hot_class) : 0;
    int32_t head = -1;

    // a long row that started in an earlier chunk: reduce its piece here
    if (rA > 0 && rpA > e0) {
        const int64_t s0 = uniform64(p.rowptr[rA - 1]);
        if (rpA - s0 > p.chunk)
            reduce_piece<T, VEC, NS, U, MSG, MAXA, IDENT, OF32>(p, rA - 1, e0, rpA < e1 ? rpA : e1, kPartial, 2 * c, lane, hot);
    }
    // rows whose first slot lies in [e0, e1) (the last chunk also takes the
    // empty rows that start at E)
    if constexpr (LIGHT) {
        const int S = kWave >> p.lg_l;
        const int sg = lane >> p.lg_l;
        int64_t rb = rA;
        while (rb < p.n_rows) {
            const int64_t rp = p.rowptr[(rb + lane) < p.n_rows ? (rb + lane) : p.n_rows];
            // rows rb .. rb+cnt-1 start in the chunk (rows starting at E are
            // empty: zero-filled separately); lane i+1 holds the end of row rb+i
            const bool in = lane < kWave - 1 && rb + lane < p.n_rows && rp < (last ? p.E : e1);
            const int cnt = __popcll(__ballot(in));
            const int64_t s_first = lane_value64(rp, 0);
            if (cnt == kWave - 1 && lane_value64(rp, kWave - 1) == s_first) {
                // 63 empty rows in a row: skip to the last row that starts at s_first
                rb = uniform_lower_bound(p.rowptr, p.n_rows + 1, s_first + 1) - 1;
                continue;
            }
            for (int i0 = 0; i0 < cnt; i0 += S) {
                const int i = i0 + sg;
                const int ii = i < cnt ? i : cnt - 1;
                const int64_t s = __shfl(rp, ii, kWave), t = __shfl(rp, ii + 1, kWave);
                const bool is_long = i < cnt && t - s > p.chunk;  // only the chunk's last row can be long
                const uint64_t lm = __ballot(is_long);
                if (lm) head = static_cast<int32_t>(rb + i0 + ((__ffsll(static_cast<unsigned long long>(lm)) - 1) >> p.lg_l));
                light_row<T, VEC, U, MSG, MAXA, IDENT, OF32>(p, rb + i, s, t, i < cnt && !is_long && t > s, lane);
            }
            if (cnt < kWave - 1) break;  // the chunk's rows end in this batch
            rb += cnt;
        }
        head = __builtin_amdgcn_readfirstlane(head);
        if (head >= 0)
            reduce_piece<T, VEC, NS, U, MSG, MAXA, IDENT, OF32>(p, head, uniform64(p.rowptr[head]), e1, kPartial, 2 * c + 1,
                                                          lane, 0);
        p.head_row[c] = head;  // uniform: every lane stores the same value (no lane-0 branch)
        return;
    }
    // rows are walked in batches of 64 row bounds; a batch that starts 63
    // empty rows (a run of them, zero-filled separately) is searched past,
    // while a shorter run is walked (each such row writes its zeros too)
    int64_t rb = rA - kWave;  // the first iteration loads the batch at rA
    int64_t rp = 0;
    for (int64_t r = rA; r < p.n_rows; ++r) {
        if (r + 1 - rb >= kWave) {
            rb = r;
            rp = p.rowptr[(rb + lane) < p.n_rows ? (rb + lane) : p.n_rows];
            const int64_t s0 = lane_value64(rp, 0);
            if (rb + kWave - 1 <= p.n_rows && lane_value64(rp, kWave - 1) == s0) {
                if (s0 >= p.E || (!last && s0 >= e1)) break;
                r = uniform64(wave_lower_bound(p.rowptr, p.n_rows + 1, s0 + 1, lane)) - 1;
                rb = r;
                rp = p.rowptr[(rb + lane) < p.n_rows ? (rb + lane) : p.n_rows];
            }
        }
        const int64_t s = uniform64(__shfl(rp, (int)(r - rb), kWave));
        const int64_t t = uniform64(__shfl(rp, (int)(r + 1 - rb), kWave));
        if (!last && s >= e1) break;
        if (t - s > p.chunk) {
            reduce_piece<T, VEC, NS, U, MSG, MAXA, IDENT, OF32>(p, r, s, e1, kPartial, 2 * c + 1, lane, hot);
            head = static_cast<int32_t>(r);
            break;
        }
        reduce_piece<T, VEC, NS, U, MSG, MAXA, IDENT, OF32>(p, r, s, t, kFull, 0, lane, hot);
    }
    p.head_row[c] = head;  // uniform: every lane stores the same value (no lane-0 branch)
}

template <typename T, bool VEC, int NS, int U, int MSG, bool MAXA, bool IDENT, bool LIGHT, bool OF32 = false>
__global__ __launch_bounds__(kBlock) void k_segment(SegParams p) {
    const int lane = threadIdx.x & (kWave - 1);
    int64_t c = uniform64((int64_t)blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave));
    if (c < p.zero_items) {  // the first work items: empty rows (short, dispatched first)
        zero_empty_rows<T, OF32>(p, c, lane);
        return;
    }
    c -= p.zero_items;
    if (p.nwin > 1) {  // all chunks of window 0, then of window 1, ...: one tail for all windows
        const int64_t w = c / p.nchunks;
        if (w >= p.nwin) return;
        c -= w * p.nchunks;
        p.fbase += w * p.fcnt;
    }
    if (c >= p.nchunks) return;
    segment_chunk_work<T, VEC, NS, U, MSG, MAXA, IDENT, LIGHT, OF32>(p, c, lane);
}

// Folding the pieces of every long row. Piece 0 is the head partial (slot
// 2c+1 of its head chunk c), piece m >= 1 the continuation in chunk c+m
// (slot 2(c+m)). The waves of a workgroup (4, or 16 for a few very long
// rows) fold contiguous, ordered ranges of the pieces with 8 (16) loads in
// flight, then wave 0 combines their results in wave order: a fixed order,
// so the fold is deterministic, and for max the earliest piece wins ties.

// The slot of piece m of the long row whose head chunk is c.
__device__ __forceinline__ int64_t piece_slot(int64_t c, int64_t m) { return m == 0 ? 2 * c + 1 : 2 * (c + m); }

// Fold pieces g0, g0 + G, g0 + 2G, ... (below K) of the long row r with head
// chunk c, in order. FINAL: write the row's result (mean divided, argmax as
// an edge id); else write the fold into the slot of piece g0 (a group's
// partial, for the second level of the grouped fold).
template <typename T, bool MAXA, int kW, int kU, bool OF32, bool FINAL = true>
__device__ __forceinline__ void fold_long_row(const SegParams &p, int64_t c, int64_t r, float (&sv)[kW][kWave],
                                              int32_t (&sp)[kW][kWave], int64_t g0 = 0, int64_t G = 1,
                                              int64_t gend = -1) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t s = p.rowptr[r], t = p.rowptr[r + 1];
    const int64_t Kall = (t - 1) / p.chunk - c + 1;  // pieces of this row
    const int64_t pend = gend < 0 ? Kall : (gend < Kall ? gend : Kall);
    const int64_t K = (pend - g0 + G - 1) / G;  // pieces folded here: g0 + G * [0, K)
    const int64_t m0 = K * wave / kW, m1 = K * (wave + 1) / kW;
    T *out = static_cast<T *>(p.out);
    for (int64_t fg = 0; fg < p.fcnt; fg += kWave) {
        const int64_t f = p.fbase + fg + lane;
        const bool on = fg + lane < p.fcnt;
        float v = 0.f;
        int32_t ps = -1;
        for (int64_t m = m0; m < m1; m += kU) {
            float o[kU];
            int32_t op[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int64_t mm = m + u;
                const int64_t slot = piece_slot(c, g0 + G * mm);
                const bool ok = on && mm < m1;
                o[u] = ok ? p.part_val[slot * p.F + f] : 0.f;
                op[u] = (ok && MAXA) ? p.part_pos[slot * p.F + f] : -1;
            }
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                if (m + u >= m1) break;
                if constexpr (MAXA) {
                    if (ps < 0 || o[u] > v) {  // later pieces hold later slots: strict > keeps the earliest
                        v = o[u];
                        ps = op[u];
                    }
                } else {
                    v += o[u];
                }
            }
        }
        sv[wave][lane] = v;
        sp[wave][lane] = ps;
        __syncthreads();
        if (wave == 0 && on) {
            float acc = sv[0][lane];
            int32_t pos = sp[0][lane];
#pragma unroll
            for (int w = 1; w < kW; ++w) {
                const float o = sv[w][lane];
                const int32_t op = sp[w][lane];
                if constexpr (MAXA) {
                    if (op >= 0 && (pos < 0 || o > acc)) {
                        acc = o;
                        pos = op;
                    }
                } else if (K * (w + 1) / kW > K * w / kW) {  // skip waves that folded no piece
                    acc += o;
                }
            }
            if constexpr (!FINAL) {
                const int64_t slot = piece_slot(c, g0);
                p.part_val[slot * p.F + f] = acc;
                if constexpr (MAXA) p.part_pos[slot * p.F + f] = pos;
            } else {
                if (!MAXA && p.mean) acc = acc / static_cast<float>(t - s);
                if constexpr (OF32) static_cast<float *>(p.out)[r * p.F + f] = acc;
                else if constexpr (sizeof(T) == 2) out[r * p.F + f] = f32_to_bf16_rne(acc);
                else out[r * p.F + f] = acc;
                if constexpr (MAXA) p.argmax[r * p.F + f] = p.perm ? p.perm[pos] : static_cast<int64_t>(pos);
            }
        }
        __syncthreads();
    }
}

// Pieces per group of the grouped fold (few, very long rows).
constexpr int64_t kFoldGroup = 64;

// Level 1 of the grouped fold: workgroup c folds, in order, the group of
// kFoldGroup pieces that starts at chunk c, of the long row chunk c
// continues and of the long row that starts in it (if they have more than
// kFoldGroup pieces), into the group's first piece slot. One workgroup on one
// CU folding all 3,640 pieces of the large graph's whole-graph pool was held
// to that CU's load bandwidth (63 us); the groups spread over the chip.
template <typename T, bool MAXA, bool OF32>
__global__ __launch_bounds__(kBlock) void k_segment_fold_groups(SegParams p) {
    __shared__ float sv[kBlock / kWave][kWave];
    __shared__ int32_t sp[kBlock / kWave][kWave];
    const int64_t c = blockIdx.x;
    if (c >= p.nchunks || p.n_rows <= 0) return;
    const int64_t e0 = c * p.chunk;
    // the row holding the chunk's first slot: the last r with rowptr[r] <= e0
    int64_t lo = 0, hi = p.n_rows - 1;
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (p.rowptr[mid] <= e0) lo = mid;
        else hi = mid - 1;
    }
    const int64_t r1 = lo, s1 = p.rowptr[r1], t1 = p.rowptr[r1 + 1];
    const int64_t h1 = s1 / p.chunk;  // its head chunk
    if (h1 < c && t1 > e0 && t1 - s1 > p.chunk && (t1 - 1) / p.chunk - h1 + 1 > kFoldGroup && (c - h1) % kFoldGroup == 0)
        fold_long_row<T, MAXA, kBlock / kWave, 8, OF32, false>(p, h1, r1, sv, sp, c - h1, 1, c - h1 + kFoldGroup);
    const int64_t r2 = p.head_row[c];
    if (r2 >= 0 && (p.rowptr[r2 + 1] - 1) / p.chunk - c + 1 > kFoldGroup)
        fold_long_row<T, MAXA, kBlock / kWave, 8, OF32, false>(p, c, r2, sv, sp, 0, 1, kFoldGroup);
}

// The fold proper: one workgroup per chunk that starts a long row. GROUPED
// (after k_segment_fold_groups): a row of more than kFoldGroup pieces folds
// its groups' partials, pieces 0, kFoldGroup, 2 kFoldGroup, ... in order.
template <typename T, bool MAXA, int WAVES, bool OF32, bool GROUPED>
__global__ __launch_bounds__(WAVES * kWave) void k_segment_fixup(SegParams p) {
    constexpr int kW = WAVES;
    constexpr int kU = WAVES > 4 ? 16 : 8;
    __shared__ float sv[kW][kWave];
    __shared__ int32_t sp[kW][kWave];
    const int64_t c = blockIdx.x;
    if (c >= p.nchunks) return;
    const int64_t r = p.head_row[c];
    if (r < 0) return;  // uniform over the workgroup
    const int64_t K = (p.rowptr[r + 1] - 1) / p.chunk - c + 1;
    if (GROUPED && K > kFoldGroup) fold_long_row<T, MAXA, kW, kU, OF32>(p, c, r, sv, sp, 0, kFoldGroup);
    else fold_long_row<T, MAXA, kW, kU, OF32>(p, c, r, sv, sp);
}

// Degree class of every row, and their histogram (hist must start at zero).
__global__ __launch_bounds__(kBlock) void k_degree_classes(const int64_t *__restrict__ rowptr, int64_t n_rows,
                                                           uint8_t *__restrict__ node_class, int32_t *__restrict__ hist) {
    __shared__ int32_t h[kClasses];
    for (int i = threadIdx.x; i < kClasses; i += kBlock) h[i] = 0;
    __syncthreads();
    for (int64_t r = blockIdx.x * (int64_t)kBlock + threadIdx.x; r < n_rows; r += (int64_t)gridDim.x * kBlock) {
        const int c = deg_class(rowptr[r + 1] - rowptr[r]);
        node_class[r] = static_cast<uint8_t>(c);
        atomicAdd(&h[c], 1);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kClasses; i += kBlock)
        if (h[i]) atomicAdd(&hist[i], h[i]);
}

// Smallest class c >= 1 such that the rows of classes >= c number at most
// `budget_rows` (the count only grows as c falls, so that c is where it
// first exceeds the budget); 0 (no hint) when every row fits or no class
// does. One wavefront: lane l holds classes 4l .. 4l+3, a suffix scan over
// the lanes gives each class its count of rows at or above it.
__global__ void k_pick_hot_class(const int32_t *__restrict__ hist, int64_t budget_rows, int32_t *__restrict__ hot) {
    static_assert(kClasses == 4 * kWave, "four classes per lane");
    const int lane = threadIdx.x;
    if (blockIdx.x != 0 || lane >= kWave) return;
    int64_t h[4], mine = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) mine += (h[i] = hist[4 * lane + i]);
    long long incl = mine;  // sum over lanes >= lane
    for (int off = 1; off < kWave; off <<= 1) {
        const long long y = __shfl_down(incl, off, kWave);
        if (lane + off < kWave) incl += y;
    }
    int64_t suf = incl - mine;  // rows of the classes above this lane's
    int first = kClasses;
#pragma unroll
    for (int i = 3; i >= 0; --i) {
        suf += h[i];
        const int c = 4 * lane + i;
        if (c >= 1 && suf <= budget_rows) first = c;
    }
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const int o = __shfl_xor(first, off, kWave);
        first = o < first ? o : first;
    }
    if (lane == 0) *hot = (first == kClasses || first <= 1) ? 0 : first;
}

// No slots at all: every row is empty (0, and the sentinel for argmax).
template <typename T>
__global__ void k_empty_rows(T *__restrict__ out, int64_t *__restrict__ argmax, int64_t n, int64_t sentinel) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        out[i] = T(0);
        if (argmax) argmax[i] = sentinel;
    }
}

template <typename T, bool MAXA, bool OF32 = false>
int launch_fixup(const SegParams &p, hipStream_t s) {
    if (p.nchunks <= 1) return PYG_OK;
    // few, very long rows (e.g. whole-graph pooling): groups of pieces folded
    // across the chip first, then 16 waves fold each row's group partials
    if (p.E > 16 * p.chunk * (p.n_rows > 0 ? p.n_rows : 1)) {
        k_segment_fold_groups<T, MAXA, OF32><<<static_cast<unsigned>(p.nchunks), kBlock, 0, s>>>(p);
        PYG_LAUNCH_CHECK();
        k_segment_fixup<T, MAXA, 16, OF32, true><<<static_cast<unsigned>(p.nchunks), 16 * kWave, 0, s>>>(p);
    } else {
        k_segment_fixup<T, MAXA, 4, OF32, false><<<static_cast<unsigned>(p.nchunks), kBlock, 0, s>>>(p);
    }
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

template <typename T, bool VEC, int NS, int MSG, bool MAXA, bool IDENT>
int launch_window(const SegParams &p, bool light, bool fixup, hipStream_t s) {
    constexpr int U = NS == 1 ? 8 : (NS == 2 ? 4 : 2);
    const int64_t nc = p.nchunks * (p.nwin > 1 ? p.nwin : 1) + p.zero_items;
    const unsigned grid = static_cast<unsigned>((nc + (kBlock / kWave) - 1) / (kBlock / kWave));
    if constexpr (NS == 1) {
        if (light) k_segment<T, VEC, NS, U, MSG, MAXA, IDENT, true><<<grid, kBlock, 0, s>>>(p);
        else k_segment<T, VEC, NS, U, MSG, MAXA, IDENT, false><<<grid, kBlock, 0, s>>>(p);
    } else {
        k_segment<T, VEC, NS, U, MSG, MAXA, IDENT, false><<<grid, kBlock, 0, s>>>(p);
    }
    PYG_LAUNCH_CHECK();
    return fixup ? launch_fixup<T, MAXA>(p, s) : PYG_OK;
}

template <typename T, bool VEC, int MSG, bool MAXA, bool IDENT>
int launch_ns(const SegParams &p, int ns, bool light, bool fixup, hipStream_t s) {
    if (ns == 1) return launch_window<T, VEC, 1, MSG, MAXA, IDENT>(p, light, fixup, s);
    if (ns == 2) return launch_window<T, VEC, 2, MSG, MAXA, IDENT>(p, false, fixup, s);
    return launch_window<T, VEC, 4, MSG, MAXA, IDENT>(p, false, fixup, s);
}

template <typename T, bool VEC, bool MAXA>
int launch_msg(const SegParams &p, int msg, bool ident, int ns, bool light, bool fixup, hipStream_t s) {
    if (ident) return launch_ns<T, VEC, kMsgSrc, MAXA, true>(p, ns, light, fixup, s);
    if constexpr (!MAXA) {
        if (msg == kMsgHeads) return launch_ns<T, VEC, kMsgHeads, false, false>(p, ns, light, fixup, s);
        if (msg == kMsgEdgeReluGrad) return launch_ns<T, VEC, kMsgEdgeReluGrad, false, false>(p, ns, light, fixup, s);
    }
    if (msg == kMsgEdgeAdd) return launch_ns<T, VEC, kMsgEdgeAdd, MAXA, false>(p, ns, light, fixup, s);
    if (msg == kMsgEdgeRelu) return launch_ns<T, VEC, kMsgEdgeRelu, MAXA, false>(p, ns, light, fixup, s);
    if (msg == kMsgEdgeMul) return launch_ns<T, VEC, kMsgEdgeMul, MAXA, false>(p, ns, light, fixup, s);
    if (msg == kMsgDiff) return launch_ns<T, VEC, kMsgDiff, MAXA, false>(p, ns, light, fixup, s);
    if (msg == kMsgWeighted) return launch_ns<T, VEC, kMsgWeighted, MAXA, false>(p, ns, light, fixup, s);
    if constexpr (!MAXA) {
        if (msg == kMsgGcn) return launch_ns<T, VEC, kMsgGcn, false, false>(p, ns, light, fixup, s);
    }
    return launch_ns<T, VEC, kMsgSrc, MAXA, false>(p, ns, light, fixup, s);
}

template <typename T>
int run_typed(const SegmentArgs &a, SegParams p, hipStream_t s) {
    const bool maxa = a.aggr == PYG_MAX;
    if (a.E == 0) {
        k_empty_rows<T><<<grid_for(a.n_rows * a.F, kBlock * 4), kBlock, 0, s>>>(
            static_cast<T *>(a.out), maxa ? a.argmax : nullptr, a.n_rows * a.F, a.sentinel);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    const int64_t row_bytes = a.F * (int64_t)sizeof(T);
    const bool vec = row_bytes % 16 == 0 && (reinterpret_cast<uintptr_t>(a.x) % 16) == 0 &&
                     (reinterpret_cast<uintptr_t>(a.out) % 16) == 0 &&
                     (!a.alpha || (a.C * (int64_t)sizeof(T)) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(a.edge_attr) % 16) == 0 &&
                     (reinterpret_cast<uintptr_t>(a.x_self) % 16) == 0;
    const int ep = vec ? 16 / (int)sizeof(T) : 1;
    const int64_t nvec = a.F / ep;  // lane vectors per row
    int mk = a.alpha ? kMsgHeads : (a.msg == PYG_MSG_DIFF ? kMsgDiff : (a.weight ? kMsgWeighted : kMsgSrc));
    if (a.msg == kSegMsgGcn) mk = kMsgGcn;
    if (a.msg == PYG_MSG_EDGE_ADD) mk = kMsgEdgeAdd;
    if (a.msg == PYG_MSG_EDGE_RELU) mk = kMsgEdgeRelu;
    if (a.msg == PYG_MSG_EDGE_MUL) mk = kMsgEdgeMul;
    if (a.msg == kSegMsgEdgeReluGrad) mk = kMsgEdgeReluGrad;
    const bool ident = a.col == nullptr;
    // narrow windows: gathered (not identity) source rows of one of the
    // plain messages, vector lanes, rows wider than a window, large in total
    const bool narrow = kWindowBytes > 0 && vec && !ident &&
                        (PYG_NARROW_ALL || mk == kMsgSrc || mk == kMsgWeighted || mk == kMsgDiff || mk == kMsgGcn) &&
                        row_bytes > kWindowBytes &&
                        row_bytes % kWindowBytes == 0 && a.n_rows * row_bytes >= kWindowMinBytes;
    // cache hint: only when the source rows do not fit in L2 (row in-degree as the hotness proxy)
    p.hot_class = nullptr;
    const int64_t hint_bytes = narrow && PYG_HINT_NARROW == 1 ? kWindowBytes : row_bytes;
    if (!ident && a.hint && row_bytes >= kHintMinRowBytes && a.n_rows * row_bytes > kHintMinBytes &&
        !(narrow && PYG_HINT_NARROW == 0)) {
        PYG_TRY(fill<int32_t>(p.class_hist, kClasses, 0, s));
        k_degree_classes<<<grid_for(a.n_rows, kBlock * 16, 256), kBlock, 0, s>>>(a.rowptr, a.n_rows, p.node_class,
                                                                                   p.class_hist);
        PYG_LAUNCH_CHECK();
        k_pick_hot_class<<<1, kWave, 0, s>>>(p.class_hist, kHotBudgetBytes / hint_bytes, p.hot_slot);
        PYG_LAUNCH_CHECK();
        p.hot_class = p.hot_slot;
    }
    // lane vectors covered by one launch (NS = 4, or one narrow window)
    const int64_t per_window = narrow ? kWindowBytes / 16 : 4 * kWave;
    // the first launch also zero-fills the empty rows (all features)
    set_zero_items(p, a.n_rows);
    if (narrow && PYG_WINDOWS_ONE_LAUNCH) {
        // every window is the same width (rows are a multiple of a window): one
        // launch, window-major, then the fold of the long rows over all features
        int lg = 0;
        while ((1 << lg) < per_window && lg < 6) ++lg;
        p.lg_l = lg;
        p.fbase = 0;
        p.fcnt = per_window * ep;
        p.nwin = nvec / per_window;
        const bool light = lg < 6 && a.E <= kLightMaxDegree * a.n_rows;
        int rc;
        if (mk == kMsgGcn && p.nwin > 1) {
            // GCN: window 0 forms every slot's weight and writes it (norm_out is
            // set); the later windows read those weights (stream order) instead
            // of forming them again
            SegParams q = p;
            q.nwin = 1;
            rc = launch_msg<T, true, false>(q, kMsgGcn, ident, 1, light, false, s);
            if (rc != PYG_OK) return rc;
            q = p;
            q.zero_items = 0;
            q.fbase = p.fcnt;
            q.nwin = p.nwin - 1;
            q.w = p.norm_out;
            rc = launch_msg<T, true, false>(q, kMsgWeighted, ident, 1, light, false, s);
        } else if (maxa) {
            rc = launch_msg<T, true, true>(p, mk, ident, 1, light, false, s);
        } else {
            rc = launch_msg<T, true, false>(p, mk, ident, 1, light, false, s);
        }
        if (rc != PYG_OK) return rc;
        p.nwin = 1;
        p.fbase = 0;
        p.fcnt = a.F;
        return maxa ? launch_fixup<T, true>(p, s) : launch_fixup<T, false>(p, s);
    }
    for (int64_t v0 = 0; v0 < nvec; v0 += per_window) {
        const int64_t vn = (nvec - v0) < per_window ? (nvec - v0) : per_window;
        const int ns = vn <= kWave ? 1 : (vn <= 2 * kWave ? 2 : 4);
        int lg = 0;
        while ((1 << lg) < (narrow ? vn : nvec) && lg < 6) ++lg;
        p.lg_l = lg;
        p.fbase = v0 * ep;
        p.fcnt = vn * ep;
        // light rows: short rows on average and at least two sub-groups per wavefront
        const bool light = ns == 1 && lg < 6 && a.E <= kLightMaxDegree * a.n_rows;
        // narrow windows fold their long rows together, once, below
        const bool fixup = !narrow;
        int rc;
        if (vec) rc = maxa ? launch_msg<T, true, true>(p, mk, ident, ns, light, fixup, s)
                           : launch_msg<T, true, false>(p, mk, ident, ns, light, fixup, s);
        else rc = maxa ? launch_msg<T, false, true>(p, mk, ident, ns, light, fixup, s)
                       : launch_msg<T, false, false>(p, mk, ident, ns, light, fixup, s);
        if (rc != PYG_OK) return rc;
        p.zero_items = 0;
    }
    if (narrow) {
        p.fbase = 0;
        p.fcnt = a.F;
        return maxa ? launch_fixup<T, true>(p, s) : launch_fixup<T, false>(p, s);
    }
    return PYG_OK;
}

// Folds the fp32 partial rows of the source blocks in block order:
// out[i] = sum over b of P[b*N + i] (mean: divided by deg_i, the row's slots
// over all blocks, as the unblocked kernel divides); max: the largest
// partial, equal values to the lower edge id, blocks without slots (argmax =
// sentinel) skipped. A fixed order: deterministic. F % 4 == 0. With `scale`,
// features from `scale_from` on (a multiple of 4) are multiplied by
// scale[i] in fp64 and rounded once. With `pieces` (sum and mean), a virtual
// row longer than `chunk` slots is read as the sum of its pieces (head
// partial, then one continuation per chunk, in order) instead of from P, so
// that no fix-up launch folds them first: that launch, one workgroup per
// chunk, took 47 us on the large power-law graph, nearly all of it spent on
// workgroups with nothing to fold.
template <typename T, bool MAXA>
__global__ __launch_bounds__(kBlock) void k_block_fold(const float *__restrict__ P, const int64_t *__restrict__ Parg,
                                                       const int64_t *__restrict__ rowptr, int64_t N, int64_t F,
                                                       int64_t B, int mean, int64_t sentinel, T *__restrict__ out,
                                                       int64_t *__restrict__ argmax, const double *__restrict__ scale,
                                                       int64_t scale_from, const float *__restrict__ pieces,
                                                       int64_t chunk) {
    const int64_t nq = N * F / 4;
    const int64_t NF = N * F;
    for (int64_t q = blockIdx.x * (int64_t)kBlock + threadIdx.x; q < nq; q += (int64_t)gridDim.x * kBlock) {
        const int64_t e = q * 4;  // element i * F + f of four consecutive features
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        int64_t a[4] = {sentinel, sentinel, sentinel, sentinel};
        for (int64_t b = 0; b < B; ++b) {
            float4 pv;
            int64_t s0 = 0, t0 = 0;
            if (!MAXA && pieces) {
                const int64_t r = b * N + e / F;
                s0 = rowptr[r];
                t0 = rowptr[r + 1];
            }
            if (!MAXA && pieces && t0 - s0 > chunk) {
                const int64_t c = s0 / chunk, K = (t0 - 1) / chunk - c + 1, f = e % F;
                pv = make_float4(0.f, 0.f, 0.f, 0.f);
                int64_t m = 0;
                for (; m + 4 <= K; m += 4) {  // four loads in flight, added in piece order
                    float4 w[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        w[u] = *reinterpret_cast<const float4 *>(pieces + piece_slot(c, m + u) * F + f);
#pragma unroll
                    for (int u = 0; u < 4; ++u) pv.x += w[u].x, pv.y += w[u].y, pv.z += w[u].z, pv.w += w[u].w;
                }
                for (; m < K; ++m) {
                    const float4 w = *reinterpret_cast<const float4 *>(pieces + piece_slot(c, m) * F + f);
                    pv.x += w.x, pv.y += w.y, pv.z += w.z, pv.w += w.w;
                }
            } else {
                pv = *reinterpret_cast<const float4 *>(P + b * NF + e);
            }
            const float pw[4] = {pv.x, pv.y, pv.z, pv.w};
            if constexpr (MAXA) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int64_t pa = Parg[b * NF + e + k];
                    if (pa != sentinel && (a[k] == sentinel || pw[k] > v[k] || (pw[k] == v[k] && pa < a[k]))) {
                        v[k] = pw[k];
                        a[k] = pa;
                    }
                }
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] += pw[k];
            }
        }
        if (!MAXA && scale && e % F >= scale_from) {
            const double si = scale[e / F];
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] = static_cast<float>(static_cast<double>(v[k]) * si);
        }
        if (!MAXA && mean) {
            const int64_t i = e / F;
            int64_t deg = 0;
            for (int64_t b = 0; b < B; ++b) deg += rowptr[b * N + i + 1] - rowptr[b * N + i];
            if (deg > 0) {
#pragma unroll
                for (int k = 0; k < 4; ++k) v[k] = v[k] / static_cast<float>(deg);
            }
        }
        if constexpr (sizeof(T) == 2) {
            const uint32_t lo = uint32_t(f32_to_bf16_rne(v[0])) | (uint32_t(f32_to_bf16_rne(v[1])) << 16);
            const uint32_t hi = uint32_t(f32_to_bf16_rne(v[2])) | (uint32_t(f32_to_bf16_rne(v[3])) << 16);
            *reinterpret_cast<uint2 *>(out + e) = make_uint2(lo, hi);
        } else {
            *reinterpret_cast<float4 *>(out + e) = make_float4(v[0], v[1], v[2], v[3]);
        }
        if constexpr (MAXA) {
#pragma unroll
            for (int k = 0; k < 4; ++k) argmax[e + k] = a[k];
        }
    }
}

// Source-blocked virtual rows: the ordinary chunked launch over the B * N
// virtual rows (window-major, and inside a window block-major, since the
// virtual rows of block b precede those of block b + 1), writing fp32
// partial rows. At any moment the wavefronts in flight gather from one
// source block of one feature window, a 1/B part of x's bytes per window.
constexpr int64_t kMaxBlocks = 32;  // source blocks of a blocked CSR, at most

// xs[i, f] = d_i^-1/2 * x[i, f] for the features f >= f0 (fp64 product,
// rounded once), four features per thread; F and f0 multiples of 4.
__global__ __launch_bounds__(kBlock) void k_prescale_rows(const float *__restrict__ x, const double *__restrict__ dinv,
                                                          int64_t N, int64_t F, int64_t f0, float *__restrict__ xs) {
    const int64_t per_row = (F - f0) / 4;
    const int64_t n = N * per_row;
    for (int64_t q = blockIdx.x * (int64_t)kBlock + threadIdx.x; q < n; q += (int64_t)gridDim.x * kBlock) {
        const int64_t i = q / per_row;
        const int64_t e = i * F + f0 + (q - i * per_row) * 4;
        const float4 v = *reinterpret_cast<const float4 *>(x + e);
        const double d = dinv[i];
        *reinterpret_cast<float4 *>(xs + e) =
            make_float4(static_cast<float>(v.x * d), static_cast<float>(v.y * d), static_cast<float>(v.z * d),
                        static_cast<float>(v.w * d));
    }
}

template <typename T, int MSG, bool MAXA>
int launch_blocked(const SegParams &p, bool light, hipStream_t s) {
    constexpr int U = 8;  // gathers in flight per lane, as in the unblocked kernel
    const int64_t nc = p.nchunks * (p.nwin > 1 ? p.nwin : 1) + p.zero_items;
    const unsigned grid = static_cast<unsigned>((nc + (kBlock / kWave) - 1) / (kBlock / kWave));
    if (light) k_segment<T, true, 1, U, MSG, MAXA, false, true, true><<<grid, kBlock, 0, s>>>(p);
    else k_segment<T, true, 1, U, MSG, MAXA, false, false, true><<<grid, kBlock, 0, s>>>(p);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

template <typename T>
int launch_blocked_msg(const SegParams &p, int mk, bool maxa, bool light, hipStream_t s) {
    if (maxa) {
        if (mk == kMsgDiff) return launch_blocked<T, kMsgDiff, true>(p, light, s);
        if (mk == kMsgWeighted) return launch_blocked<T, kMsgWeighted, true>(p, light, s);
        return launch_blocked<T, kMsgSrc, true>(p, light, s);
    }
    if (mk == kMsgDiff) return launch_blocked<T, kMsgDiff, false>(p, light, s);
    if (mk == kMsgWeighted) return launch_blocked<T, kMsgWeighted, false>(p, light, s);
    if (mk == kMsgGcn) return launch_blocked<T, kMsgGcn, false>(p, light, s);
    return launch_blocked<T, kMsgSrc, false>(p, light, s);
}

struct SegWs {
    float *part_val;
    int32_t *part_pos;
    int32_t *head_row;
    int32_t *class_hist;
    int32_t *hot_slot;
    uint8_t *node_class;
    size_t bytes;
};

SegWs carve_segment(void *base, int64_t E, int64_t F, int aggr, int64_t chunk, int64_t n_rows) {
    const int64_t nchunks = E > 0 ? (E + chunk - 1) / chunk : 0;
    Carver c(base);
    SegWs w{};
    w.part_val = c.take<float>(2 * nchunks * F);
    w.part_pos = c.take<int32_t>(aggr == PYG_MAX ? 2 * nchunks * F : 0);
    w.head_row = c.take<int32_t>(nchunks);
    w.class_hist = c.take<int32_t>(kClasses);
    w.hot_slot = c.take<int32_t>(1);
    w.node_class = c.take<uint8_t>(n_rows);
    w.bytes = c.used + 256;
    return w;
}

struct BlockedWs {
    float *P;        // [B * N, F] fp32 partial rows
    int64_t *Parg;   // [B * N, F] their argmax (max only)
    void *seg;       // the segment reduction's workspace over the B * N virtual rows
    size_t seg_bytes;
    size_t bytes;
};

BlockedWs carve_blocked(void *base, int64_t E, int64_t N, int64_t F, int64_t B, int aggr, int64_t chunk) {
    Carver c(base);
    BlockedWs w{};
    w.P = c.take<float>(B * N * F);
    w.Parg = c.take<int64_t>(aggr == PYG_MAX ? B * N * F : 0);
    w.seg_bytes = carve_segment(nullptr, E, F, aggr, chunk, B * N).bytes;
    w.seg = c.take<char>(w.seg_bytes);
    w.bytes = c.used + 256;
    return w;
}

}  // namespace

size_t segment_blocked_workspace(int64_t E, int64_t N, int64_t F, int64_t B, int aggr, int64_t chunk) {
    return carve_blocked(nullptr, E, N, F, B, aggr, segment_chunk(E, B * N, chunk)).bytes;
}

int segment_reduce_blocked(const SegmentArgs &a, int64_t B, void *ws, size_t ws_bytes, hipStream_t s) {
    const int64_t N = a.n_rows, F = a.F, E = a.E;
    if (N == 0 || F == 0) return PYG_OK;
    const bool maxa = a.aggr == PYG_MAX;
    const int64_t sz = a.dtype == PYG_BF16 ? 2 : 4;
    if ((F * sz) % 16 != 0 || reinterpret_cast<uintptr_t>(a.x) % 16 != 0 || reinterpret_cast<uintptr_t>(a.out) % 16 != 0)
        return PYG_ERR_UNSUPPORTED;  // 16-byte lane vectors only
    if (B < 2 || B > kMaxBlocks) return PYG_ERR_UNSUPPORTED;
    const int64_t chunk = segment_chunk(E, B * N, a.chunk);
    const BlockedWs w = carve_blocked(ws, E, N, F, B, a.aggr, chunk);
    if (!ws || ws_bytes < w.bytes) return PYG_ERR_WORKSPACE;
    if (E == 0) {
        if (a.dtype == PYG_BF16)
            k_empty_rows<uint16_t><<<grid_for(N * F, kBlock * 4), kBlock, 0, s>>>(static_cast<uint16_t *>(a.out),
                                                                                 maxa ? a.argmax : nullptr, N * F, E);
        else
            k_empty_rows<float><<<grid_for(N * F, kBlock * 4), kBlock, 0, s>>>(static_cast<float *>(a.out),
                                                                              maxa ? a.argmax : nullptr, N * F, E);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    const SegWs sw = carve_segment(w.seg, E, F, a.aggr, chunk, B * N);
    SegParams p{};
    p.x = a.x;
    p.F = F;
    p.rowptr = a.rowptr;
    p.col = a.col;
    p.w = a.weight;
    p.perm = a.perm;
    p.n_rows = B * N;
    p.E = E;
    p.chunk = chunk;
    p.nchunks = (E + chunk - 1) / chunk;
    p.mean = 0;  // partial sums; the fold divides
    p.sentinel = E;
    p.out = w.P;
    p.argmax = maxa ? w.Parg : nullptr;
    p.part_val = sw.part_val;
    p.part_pos = sw.part_pos;
    p.head_row = sw.head_row;
    p.class_hist = sw.class_hist;
    p.hot_slot = sw.hot_slot;
    p.node_class = sw.node_class;
    p.hot_class = nullptr;
    p.blocks = B;
    p.rpb = N;
    p.dinv = a.dinv;
    p.norm_out = a.norm_out;
    // windows of up to 128 bytes: 8 lanes of 16 bytes (fewer for narrower rows)
    const int64_t ep = 16 / sz, nvec = F / ep;
    int lg = 0;
    while ((1 << lg) < nvec && lg < 3) ++lg;
    p.lg_l = lg;
    p.fbase = 0;
    p.fcnt = (int64_t(1) << lg) * ep;
    p.nwin = (F + p.fcnt - 1) / p.fcnt;
    if (p.nchunks * p.nwin >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    int mk = a.msg == PYG_MSG_DIFF ? kMsgDiff : (a.weight ? kMsgWeighted : kMsgSrc);
    if (a.msg == kSegMsgGcn) mk = kMsgGcn;
    if (mk == kMsgGcn && (maxa || !a.dinv || !a.norm_out)) return PYG_ERR_INVALID_ARG;
    // short virtual rows on average: one sub-group per row
    const bool light = lg < 6 && E <= kLightMaxDegree * B * N;
    set_zero_items(p, B * N);  // the first launch zero-fills the empty virtual rows
    int rc;
    auto launch = [&](const SegParams &q, int kind) {
        return a.dtype == PYG_BF16 ? launch_blocked_msg<uint16_t>(q, kind, maxa, light, s)
                                   : launch_blocked_msg<float>(q, kind, maxa, light, s);
    };
    // GCN on fp32 rows: the windows that need no norms propagate the rows
    // d_j^-1/2 x_j (times the edge weight, if any) and the fold multiplies
    // them by d_i^-1/2 (no per-slot norm is formed there). When the caller
    // wants the norms, window 0 still forms, uses and writes them.
    const bool prescale = mk == kMsgGcn && a.dtype == PYG_F32 && a.x_scaled;
    const int64_t first_scaled = (a.norms_wanted || !prescale) ? p.fcnt : 0;  // first pre-scaled feature
    if (mk == kMsgGcn) {
        SegParams q = p;
        if (first_scaled > 0) {
            // window 0 forms every slot's weight (and writes it); without
            // pre-scaled rows the later windows read those weights back
            q.nwin = 1;
            rc = launch(q, kMsgGcn);
            if (rc != PYG_OK) return rc;
        }
        const int64_t rest = p.nwin - first_scaled / p.fcnt;  // windows after the norm-forming one
        if (rest > 0) {
            q = p;
            if (first_scaled > 0) q.zero_items = 0;  // the first launch did
            q.fbase = first_scaled;
            q.nwin = rest;
            if (prescale) {
                k_prescale_rows<<<grid_for(N * (F - first_scaled) / 4, kBlock, 1 << 16), kBlock, 0, s>>>(
                    static_cast<const float *>(a.x), a.dinv, N, F, first_scaled, a.x_scaled);
                PYG_LAUNCH_CHECK();
                q.x = a.x_scaled;
                q.w = a.weight;
                rc = launch(q, a.weight ? kMsgWeighted : kMsgSrc);
            } else {
                q.w = p.norm_out;
                rc = launch(q, kMsgWeighted);
            }
        }
    } else {
        rc = launch(p, mk);
    }
    if (rc != PYG_OK) return rc;
    // long virtual rows: their pieces (all features) folded into P by the
    // fix-up (max, and few very long rows), or for sum and mean read by the
    // block fold itself
    p.nwin = 1;
    p.fbase = 0;
    p.fcnt = F;
    const bool fold_pieces = !maxa && p.nchunks > 1 && !(p.E > 16 * p.chunk * (p.n_rows > 0 ? p.n_rows : 1));
    if (!fold_pieces) {
        if (a.dtype == PYG_BF16)
            rc = maxa ? launch_fixup<uint16_t, true, true>(p, s) : launch_fixup<uint16_t, false, true>(p, s);
        else rc = maxa ? launch_fixup<float, true, true>(p, s) : launch_fixup<float, false, true>(p, s);
        if (rc != PYG_OK) return rc;
    }
    const float *pieces = fold_pieces ? p.part_val : nullptr;
    const unsigned g = grid_for(N * F / 4, kBlock, 1 << 16);
    const int mean = a.aggr == PYG_MEAN;
    const double *scale = prescale ? a.dinv : nullptr;
    const int64_t scale_from = first_scaled;
    if (a.dtype == PYG_BF16) {
        if (maxa) k_block_fold<uint16_t, true><<<g, kBlock, 0, s>>>(w.P, w.Parg, a.rowptr, N, F, B, mean, E,
                                                                      static_cast<uint16_t *>(a.out), a.argmax,
                                                                      nullptr, 0, nullptr, 0);
        else k_block_fold<uint16_t, false><<<g, kBlock, 0, s>>>(w.P, w.Parg, a.rowptr, N, F, B, mean, E,
                                                                  static_cast<uint16_t *>(a.out), a.argmax, nullptr, 0,
                                                                  pieces, p.chunk);
    } else {
        if (maxa) k_block_fold<float, true><<<g, kBlock, 0, s>>>(w.P, w.Parg, a.rowptr, N, F, B, mean, E,
                                                                   static_cast<float *>(a.out), a.argmax, nullptr, 0,
                                                                   nullptr, 0);
        else k_block_fold<float, false><<<g, kBlock, 0, s>>>(w.P, w.Parg, a.rowptr, N, F, B, mean, E,
                                                               static_cast<float *>(a.out), a.argmax, scale,
                                                               scale_from, pieces, p.chunk);
    }
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

int64_t segment_chunk(int64_t E, int64_t n_rows, int64_t requested) {
    if (requested > 0) return requested;
    int64_t c;
    if (n_rows > 0 && E <= kLightMaxDegree * n_rows) {
        // short rows: about 16 rows per wavefront
        const int64_t avg = (E + n_rows - 1) / n_rows;
        c = 16;
        while (c < 16 * avg && c < 2048) c <<= 1;
        // small graphs: enough wavefronts to fill the chip (long rows are
        // left alone: smaller chunks only add pieces to fold)
        while (c > 16 && E < c * (int64_t)PYG_MIN_CHUNKS) c >>= 1;
    } else {
        // long rows: grow with E up to PYG_SEG_MAX_CHUNK slots (the large
        // power-law graph: 2048 -> 1024 took the propagate 5.28 -> 5.21 ms,
        // a shorter drain tail at the end of the launch)
        c = 64;
        while (c < PYG_SEG_MAX_CHUNK && c * 32768 < E) c <<= 1;
    }
    return c;
}

size_t segment_workspace(int64_t E, int64_t F, int aggr, int64_t chunk, int64_t n_rows) {
    return carve_segment(nullptr, E, F, aggr, segment_chunk(E, n_rows, chunk), n_rows).bytes;
}

int segment_reduce(const SegmentArgs &a, void *ws, size_t ws_bytes, hipStream_t s) {
    if (a.n_rows == 0 || a.F == 0) return PYG_OK;
    const int64_t chunk = segment_chunk(a.E, a.n_rows, a.chunk);
    const SegWs w = carve_segment(ws, a.E, a.F, a.aggr, chunk, a.n_rows);
    if (ws_bytes < w.bytes || !ws) return PYG_ERR_WORKSPACE;
    SegParams p{};
    p.x = a.x;
    p.F = a.F;
    p.rowptr = a.rowptr;
    p.col = a.col;
    p.w = a.weight;
    p.alpha = a.alpha;
    p.alpha_idx = a.alpha_idx;
    p.ea = a.edge_attr;
    p.ea_perm = a.attr_perm;
    p.ea_idx = a.attr_idx;
    p.x_self = a.x_self;
    p.H = a.H;
    p.C = a.C;
    p.perm = a.perm;
    p.n_rows = a.n_rows;
    p.E = a.E;
    p.chunk = chunk;
    p.nchunks = a.E > 0 ? (a.E + chunk - 1) / chunk : 0;
    p.mean = a.aggr == PYG_MEAN;
    p.sentinel = a.sentinel;
    p.out = a.out;
    p.argmax = a.argmax;
    p.part_val = w.part_val;
    p.part_pos = w.part_pos;
    p.head_row = w.head_row;
    p.class_hist = w.class_hist;
    p.hot_slot = w.hot_slot;
    p.node_class = w.node_class;
    p.dinv = a.dinv;
    p.norm_out = a.norm_out;
    return a.dtype == PYG_BF16 ? run_typed<uint16_t>(a, p, s) : run_typed<float>(a, p, s);
}

}  // namespace pyg
