// Shared device/host helpers of the gfx950 propagate library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "pyg_mi355x.h"

namespace pyg {

constexpr int kWave = 64;   // CDNA wavefront width
constexpr int kBlock = 256; // threads per workgroup for every kernel (4 waves)

#define PYG_LAUNCH_CHECK()                                      \
    do {                                                        \
        if (hipGetLastError() != hipSuccess) return PYG_ERR_HIP; \
    } while (0)

#define PYG_TRY(expr)                  \
    do {                               \
        int _rc = (expr);              \
        if (_rc != PYG_OK) return _rc; \
    } while (0)

static inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Carves aligned sub-buffers out of one caller workspace.
struct Carver {
    char *base;
    size_t used = 0;
    explicit Carver(void *p) : base(static_cast<char *>(p)) {}
    template <typename T>
    T *take(size_t count) {
        used = align_up(used, 256);
        T *p = reinterpret_cast<T *>(base ? base + used : nullptr);
        used += count * sizeof(T);
        return p;
    }
};

static inline unsigned grid_for(int64_t work, int64_t per_block, int64_t cap = 1 << 20) {
    int64_t g = (work + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return static_cast<unsigned>(g);
}

// ---------------------------------------------------------------- numerics

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// fp32 -> bf16 with round-to-nearest-even (inputs are finite).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Monotone map of finite floats to uint32 (a < b  <=>  key(a) < key(b)).
__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float order_key_inv(uint32_t k) {
    uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// -0.0 -> +0.0 so that zeros tie when comparing for max.
__device__ __forceinline__ float canon_zero(float m) { return m == 0.0f ? 0.0f : m; }

// ---------------------------------------------------------- wave helpers

// A wave-uniform 64-bit value in scalar registers.
__device__ __forceinline__ int64_t uniform64(int64_t v) {
    const uint64_t u = static_cast<uint64_t>(v);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
    return static_cast<int64_t>((uint64_t(hi) << 32) | lo);
}

// The 64-bit value that lane l holds, read into scalar registers.
__device__ __forceinline__ int64_t lane_value64(int64_t v, int l) {
    const uint64_t u = static_cast<uint64_t>(v);
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(u), l);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(u >> 32), l);
    return static_cast<int64_t>((uint64_t(hi) << 32) | lo);
}

// First index i in [0, len) with a[i] >= key; a is non-decreasing and
// a[len - 1] >= key. 64-ary search: one coalesced probe per lane per level.
__device__ inline int64_t wave_lower_bound(const int64_t *__restrict__ a, int64_t len, int64_t key, int lane) {
    int64_t lo = 0, hi = len;
    while (hi - lo > kWave) {
        const int64_t step = (hi - lo + kWave - 1) / kWave;
        int64_t idx = lo + (int64_t)(lane + 1) * step - 1;
        if (idx > hi - 1) idx = hi - 1;
        const uint64_t m = __ballot(a[idx] >= key);
        if (m == 0) return len - 1;  // not monotone: malformed input, stay in bounds
        const int lf = __ffsll(static_cast<unsigned long long>(m)) - 1;
        const int64_t nhi = lo + (int64_t)(lf + 1) * step;
        lo = lo + (int64_t)lf * step;
        hi = nhi < hi ? nhi : hi;
    }
    const int64_t idx = lo + lane;
    const uint64_t m = __ballot(idx >= hi || a[idx] >= key);
    return m ? lo + (__ffsll(static_cast<unsigned long long>(m)) - 1) : len - 1;
}

// First index i in [0, len) with a[i] >= key (a non-decreasing, a[len - 1] >=
// key), by a plain binary search on wave-uniform values: about log2(len)
// dependent loads but almost no vector registers, for searches that are rare
// (skipping a long run of empty rows) inside kernels whose occupancy is set
// by their register use.
__device__ inline int64_t uniform_lower_bound(const int64_t *__restrict__ a, int64_t len, int64_t key) {
    int64_t lo = 0, hi = len - 1;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (uniform64(a[mid]) >= key) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}

// The next row of a walk over a chunk's slots, after row r that ends at slot
// t < E: row r + 1, or when a long run of empty rows follows, the row that
// holds slot t.
// A run of empty rows all starts at t, so it belongs to one chunk; stepping
// through it row by row made that chunk's wavefront the whole call's tail.
__device__ __forceinline__ int64_t next_row_with_slots(const int64_t *__restrict__ rowptr, int64_t N, int64_t r,
                                                       int64_t t, int lane) {
    if (uniform64(rowptr[r + 2]) != t) return r + 1;  // r + 2 <= N: row r + 1 exists, as t < rowptr[N]
    // a few empty rows are stepped through; a run of 32 or more is searched past
    if (uniform64(rowptr[(r + 33) < N ? (r + 33) : N]) != t) return r + 1;
    return uniform_lower_bound(rowptr, N + 1, t + 1) - 1;
}

// Workgroups of a launch are dealt to the 8 XCDs in turn (workgroup w runs
// on XCD w % 8). xcd_major(w, T) renumbers the T workgroups so that each XCD
// takes one contiguous range of the new order: work items that are
// neighbours in that order (and share data or cache lines) share one XCD's
// L2. A bijection of [0, T) for every T; placement only, never results.
constexpr int kXcds = 8;
__device__ __forceinline__ int64_t xcd_major(int64_t w, int64_t T) {
    const int64_t q = T / kXcds, rem = T % kXcds, xcd = w % kXcds, wi = w / kXcds;
    return xcd < rem ? xcd * (q + 1) + wi : rem * (q + 1) + (xcd - rem) * q + wi;
}

// ------------------------------------------------------------ small kernels

template <typename T>
__global__ void k_fill(T *__restrict__ p, int64_t n, T v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

template <typename T>
static inline int fill(T *p, int64_t n, T v, hipStream_t s) {
    if (n <= 0) return PYG_OK;
    k_fill<T><<<grid_for(n, kBlock * 4), kBlock, 0, s>>>(p, n, v);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

// ---------------------------------------------------------- internal API

// Exclusive (or inclusive) prefix sum of n elements; `in` may equal `out`.
// Scratch: scan_workspace_elems(n) elements of T.
size_t scan_workspace_elems(int64_t n);
int scan_u32(const uint32_t *in, uint32_t *out, int64_t n, bool inclusive, uint32_t *ws, hipStream_t s);
int scan_i64(const int64_t *in, int64_t *out, int64_t n, bool inclusive, int64_t *ws, hipStream_t s);

// In-degree histograms (LDS-sliced, deterministic); scratch degree_workspace(E, N) bytes.
size_t degree_workspace(int64_t E, int64_t N);
int count_targets_i64(const int64_t *dst, int64_t E, int64_t N, int64_t *out, void *ws, hipStream_t s);
int count_targets_f64(const int64_t *dst, int64_t E, int64_t N, double *out, void *ws, hipStream_t s);

// Target-sorted segment reduction shared by propagate (CSR) and pooling.
struct SegmentArgs {
    const void *x;      // source rows [n_src, F]
    int dtype;
    int64_t F;
    const int64_t *rowptr; // [n_rows + 1]
    const int32_t *col;    // [E] source row per slot; NULL = identity (slot id)
    const float *weight;   // [E] or NULL
    const float *alpha;    // [E, H] per-head weights in slot order, or NULL (sum only)
    const int32_t *alpha_idx;  // [E] row of alpha for each slot, or NULL (row = slot)
    const void *edge_attr;       // [E, F] edge features in x's dtype (edge messages), or NULL
    const int64_t *attr_perm;    // non-NULL: edge_attr rows are COO edge ids, reached through perm
    const int32_t *attr_idx;     // non-NULL: edge_attr row attr_idx[slot] (precedence over attr_perm)
    const void *x_self;          // kSegMsgEdgeReluGrad: the rows' own features [n_rows, F]
    int64_t H;             // heads; feature f belongs to head f / C
    int64_t C;
    const int64_t *perm;   // [E] id reported by argmax; NULL = slot id
    int64_t n_rows;
    int64_t E;
    int msg;
    int aggr;
    int64_t chunk;
    int64_t sentinel;   // argmax of an empty row
    void *out;          // [n_rows, F]
    int64_t *argmax;    // [n_rows, F] or NULL
    bool hint;          // allow the cache-policy hint for hub source rows
    const double *dinv; // kSegMsgGcn: d^-1/2 of every row [n_rows]
    float *norm_out;    // kSegMsgGcn: the slots' weights written here [E], or NULL
    float *x_scaled;    // kSegMsgGcn, blocked, fp32 x: room for d^-1/2 x [n_rows, F], or NULL
    bool norms_wanted;  // kSegMsgGcn, blocked: the caller asked for the norms (norm_out is theirs)
};
// Internal message kind beyond pyg_msg (sum only): the backward of
// max(x_j + e, 0) over the reversed graph, x = the scaled upstream gradient,
// gate x_self[row] + e > 0.
constexpr int kSegMsgEdgeReluGrad = 100;
// Internal message kind (sum only): GCN, slot weight dinv[col] * w * dinv[row]
// formed in fp64 and rounded once (w = csr weight, or 1), optionally written out.
constexpr int kSegMsgGcn = 101;
int64_t segment_chunk(int64_t E, int64_t n_rows, int64_t requested);
// Source-blocked form: a.rowptr has B * n_rows + 1 entries (virtual row
// b * n_rows + i = the slots of target i whose source lies in block b), a.col,
// a.weight and a.perm are in that slot order; 2 <= B <= 32, 16-byte rows.
// Plain, weighted and difference messages, any aggregation; GCN messages
// (sum).
size_t segment_blocked_workspace(int64_t E, int64_t n_rows, int64_t F, int64_t B, int aggr, int64_t chunk);
int segment_reduce_blocked(const SegmentArgs &a, int64_t B, void *ws, size_t ws_bytes, hipStream_t s);
size_t segment_workspace(int64_t E, int64_t F, int aggr, int64_t chunk, int64_t n_rows);
int segment_reduce(const SegmentArgs &a, void *ws, size_t ws_bytes, hipStream_t s);

// inv[perm[p]] = p for a CSR's slot -> edge-id permutation (ids outside
// [0, E) skipped); transpose_map: map_t[q] = the csr slot of the edge in
// slot q of csr_t (inv: E int32 of scratch).
int inverse_perm(const int64_t *perm, int64_t E, int32_t *inv, hipStream_t s);
int transpose_map(const pyg_csr *csr, const pyg_csr *csr_t, int32_t *inv, int32_t *map_t, hipStream_t s);
// The same inverse with coalesced writes (a radix partition of the (id, slot)
// pairs by the id's high bits, then one LDS block of ids per workgroup);
// scratch inverse_perm_sorted_workspace(E) bytes.
size_t inverse_perm_sorted_workspace(int64_t E);
int inverse_perm_sorted(const int64_t *perm, int64_t E, int32_t *inv, void *ws, size_t ws_bytes, hipStream_t s);

// Every argument check of pyg_propagate (nothing is launched); on success
// *need is the workspace the call takes.
int propagate_check(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                    const float *edge_weight, const pyg_csr *csr, int msg, int aggr, int kernel, const void *out,
                    const int64_t *argmax, size_t *need);

// Unsorted-COO gather/scatter with hardware atomics.
size_t coo_workspace(int dtype, int64_t N, int64_t F, int aggr);
// ea: [E, F] edge features in x's dtype for the edge messages, else NULL.
int coo_propagate(const void *x, int dtype, int64_t N, int64_t F, const int64_t *ei, int64_t E, const float *w, int msg,
                  int aggr, void *out, int64_t *argmax, void *ws, size_t ws_bytes, hipStream_t s,
                  const void *ea = nullptr);

}  // namespace pyg
