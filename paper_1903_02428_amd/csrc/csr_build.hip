// Preprocessing: in-degree, stable COO -> target-sorted CSR, index validation.
//
// The CSR is the row-ordered ("coalesced") layout that Appendix A says a
// sparse-matrix product needs and that should be built once, as
// preprocessing. Here it is built on the GPU with a stable LSD radix sort of
// the target ids (digit-major tile histograms, a device scan, then a
// tile-ordered scatter that ranks equal digits with wavefront ballots), so
// the slots of a row keep ascending COO edge id and the result is unique.
#include "common.hpp"

namespace pyg {
namespace {

constexpr int kTileItems = 16;
constexpr int64_t kTile = (int64_t)kBlock * kTileItems;  // elements per radix tile
constexpr int kMaxDigitBits = 8;

__global__ void k_count_targets(const int64_t *__restrict__ dst, int64_t E, unsigned long long *__restrict__ cnt) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < E; k += (int64_t)gridDim.x * blockDim.x)
        atomicAdd(&cnt[dst[k]], 1ull);
}

__device__ __forceinline__ uint32_t load_key(const int64_t *dst64, const uint32_t *keys, int64_t i) {
    return dst64 ? static_cast<uint32_t>(dst64[i]) : keys[i];
}

__global__ __launch_bounds__(kBlock) void k_radix_hist(const int64_t *__restrict__ dst64, const uint32_t *__restrict__ keys,
                                                       int64_t E, int shift, int bits, int64_t ntiles,
                                                       uint32_t *__restrict__ hist) {
    __shared__ uint32_t h[1 << kMaxDigitBits];
    const int radix = 1 << bits;
    const uint32_t mask = radix - 1;
    for (int i = threadIdx.x; i < radix; i += kBlock) h[i] = 0;
    __syncthreads();
    const int64_t tile = blockIdx.x;
    const int64_t base = tile * kTile + threadIdx.x;
#pragma unroll 4
    for (int r = 0; r < kTileItems; ++r) {
        const int64_t i = base + (int64_t)r * kBlock;
        if (i < E) atomicAdd(&h[(load_key(dst64, keys, i) >> shift) & mask], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < radix; i += kBlock) hist[(int64_t)i * ntiles + tile] = h[i];
}

// Stable scatter of one tile. Elements are visited in rounds of kBlock
// consecutive ids (round r, thread t -> id tile*kTile + r*kBlock + t), which is
// id order; inside a round, equal digits are ranked by wavefront ballots and
// then by wave index, so every element lands after all earlier equal digits.
__global__ __launch_bounds__(kBlock) void k_radix_scatter(
    const int64_t *__restrict__ dst64, const uint32_t *__restrict__ keys_in, const uint32_t *__restrict__ vals_in,
    int64_t E, int shift, int bits, int64_t ntiles, const uint32_t *__restrict__ offsets,
    uint32_t *__restrict__ keys_out, uint32_t *__restrict__ vals_out,
    int64_t *__restrict__ perm, int32_t *__restrict__ col, const int64_t *__restrict__ src64,
    float *__restrict__ wcsr, const float *__restrict__ w) {
    constexpr int kWaves = kBlock / kWave;
    __shared__ uint32_t run[1 << kMaxDigitBits];
    __shared__ uint32_t cnt[kWaves][1 << kMaxDigitBits];
    const int radix = 1 << bits;
    const uint32_t mask = radix - 1;
    const int64_t tile = blockIdx.x;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int i = threadIdx.x; i < radix; i += kBlock) run[i] = offsets[(int64_t)i * ntiles + tile];
    for (int r = 0; r < kTileItems; ++r) {
        const int64_t i = tile * kTile + (int64_t)r * kBlock + threadIdx.x;
        const bool valid = i < E;
        uint32_t key = 0, val = 0;
        if (valid) {
            key = load_key(dst64, keys_in, i);
            val = vals_in ? vals_in[i] : static_cast<uint32_t>(i);
        }
        const uint32_t d = (key >> shift) & mask;
        for (int t = threadIdx.x; t < kWaves * radix; t += kBlock) (&cnt[0][0])[(t / radix) * (1 << kMaxDigitBits) + (t % radix)] = 0;
        __syncthreads();
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < bits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        const uint32_t rank = __popcll(peers & lt_mask);
        if (valid && rank == 0) cnt[wave][d] = __popcll(peers);
        __syncthreads();
        for (int t = threadIdx.x; t < radix; t += kBlock) {
            uint32_t acc = run[t];
#pragma unroll
            for (int wv = 0; wv < kWaves; ++wv) {
                const uint32_t c = cnt[wv][t];
                cnt[wv][t] = acc;
                acc += c;
            }
            run[t] = acc;
        }
        __syncthreads();
        if (valid) {
            const uint32_t pos = cnt[wave][d] + rank;
            if (perm) {
                perm[pos] = val;
                col[pos] = static_cast<int32_t>(src64[val]);
                if (wcsr) wcsr[pos] = w[val];
            } else {
                keys_out[pos] = key;
                vals_out[pos] = val;
            }
        }
        __syncthreads();
    }
}

// N <= 1: every edge targets node 0, the CSR order is the COO order.
__global__ void k_identity_csr(const int64_t *__restrict__ src, int64_t E, int64_t *__restrict__ perm,
                               int32_t *__restrict__ col, float *__restrict__ wcsr, const float *__restrict__ w) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < E; k += (int64_t)gridDim.x * blockDim.x) {
        perm[k] = k;
        col[k] = static_cast<int32_t>(src[k]);
        if (wcsr) wcsr[k] = w[k];
    }
}

__global__ void k_validate_coo(const int64_t *__restrict__ ei, int64_t n, int64_t N, unsigned long long *__restrict__ bad) {
    unsigned long long local = 0;
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n; k += (int64_t)gridDim.x * blockDim.x)
        local += (ei[k] < 0 || ei[k] >= N);
    if (local) atomicAdd(bad, local);
}

__global__ void k_validate_batch(const int64_t *__restrict__ b, int64_t N, int64_t B, unsigned long long *__restrict__ bad) {
    unsigned long long local = 0;
    for (int64_t n = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; n < N; n += (int64_t)gridDim.x * blockDim.x)
        local += (b[n] < 0 || b[n] >= B || (n > 0 && b[n] < b[n - 1]));
    if (local) atomicAdd(bad, local);
}

int digit_plan(int64_t N, int *passes, int *bits_per_pass) {
    int nb = 0;
    while (nb < 63 && (int64_t(1) << nb) < N) ++nb;  // bits of N-1
    *passes = (nb + kMaxDigitBits - 1) / kMaxDigitBits;
    *bits_per_pass = *passes ? (nb + *passes - 1) / *passes : 0;
    return nb;
}

struct CsrWs {
    uint32_t *keys[2];
    uint32_t *vals[2];
    uint32_t *hist;
    uint32_t *hist_scan;
    int64_t *row_scan;
    size_t bytes;
};

CsrWs carve_csr(void *base, int64_t E, int64_t N) {
    int passes, bpp;
    digit_plan(N, &passes, &bpp);
    const int64_t ntiles = (E + kTile - 1) / kTile;
    const int64_t nhist = ntiles << (passes ? bpp : 0);
    Carver c(base);
    CsrWs w{};
    const int64_t bufs = passes >= 2 ? E : 0;
    for (int i = 0; i < 2; ++i) {
        w.keys[i] = c.take<uint32_t>(i == 0 || passes >= 3 ? bufs : 0);
        w.vals[i] = c.take<uint32_t>(i == 0 || passes >= 3 ? bufs : 0);
    }
    w.hist = c.take<uint32_t>(nhist);
    w.hist_scan = c.take<uint32_t>(scan_workspace_elems(nhist));
    w.row_scan = c.take<int64_t>(scan_workspace_elems(N));
    w.bytes = c.used + 256;
    return w;
}

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" int pyg_degree(const int64_t *edge_index, int64_t E, int64_t N, int64_t *deg, void *stream) {
    if (E < 0 || N < 0 || (E > 0 && !edge_index) || (N > 0 && !deg)) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (E > 0 && N == 0) return PYG_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    PYG_TRY(fill<int64_t>(deg, N, 0, s));
    if (E == 0) return PYG_OK;
    k_count_targets<<<grid_for(E, kBlock * 8), kBlock, 0, s>>>(edge_index + E, E, reinterpret_cast<unsigned long long *>(deg));
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

extern "C" int pyg_coo_to_csr_workspace(int64_t E, int64_t N, size_t *bytes) {
    if (E < 0 || N < 0 || !bytes) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve_csr(nullptr, E, N).bytes;
    return PYG_OK;
}

extern "C" int pyg_coo_to_csr(const int64_t *edge_index, int64_t E, int64_t N, const float *edge_weight,
                              int64_t *rowptr, int32_t *col, int64_t *perm, float *weight_csr,
                              void *ws, size_t ws_bytes, void *stream) {
    if (E < 0 || N < 0 || !rowptr) return PYG_ERR_INVALID_ARG;
    if (E > 0 && (!edge_index || !col || !perm || N == 0)) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (!edge_weight) weight_csr = nullptr;
    const CsrWs w = carve_csr(ws, E, N);
    if (ws_bytes < w.bytes || (w.bytes > 256 && !ws)) return PYG_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;

    // row pointers: count per target into rowptr[1..N], inclusive scan in place
    PYG_TRY(fill<int64_t>(rowptr, N + 1, 0, s));
    if (E == 0) return PYG_OK;
    k_count_targets<<<grid_for(E, kBlock * 8), kBlock, 0, s>>>(dst, E, reinterpret_cast<unsigned long long *>(rowptr + 1));
    PYG_LAUNCH_CHECK();
    PYG_TRY(scan_i64(rowptr + 1, rowptr + 1, N, true, w.row_scan, s));

    int passes, bpp;
    const int nb = digit_plan(N, &passes, &bpp);
    if (passes == 0) {
        k_identity_csr<<<grid_for(E, kBlock * 4), kBlock, 0, s>>>(src, E, perm, col, weight_csr, edge_weight);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    const int64_t ntiles = (E + kTile - 1) / kTile;
    const uint32_t *kin = nullptr, *vin = nullptr;
    int shift = 0;
    for (int p = 0; p < passes; ++p) {
        const int bits = (nb - shift) < bpp ? (nb - shift) : bpp;
        const bool last = p == passes - 1;
        const int64_t nhist = ntiles << bits;
        k_radix_hist<<<(unsigned)ntiles, kBlock, 0, s>>>(p == 0 ? dst : nullptr, kin, E, shift, bits, ntiles, w.hist);
        PYG_LAUNCH_CHECK();
        PYG_TRY(scan_u32(w.hist, w.hist, nhist, false, w.hist_scan, s));
        uint32_t *kout = last ? nullptr : w.keys[p & 1];
        uint32_t *vout = last ? nullptr : w.vals[p & 1];
        k_radix_scatter<<<(unsigned)ntiles, kBlock, 0, s>>>(
            p == 0 ? dst : nullptr, kin, vin, E, shift, bits, ntiles, w.hist, kout, vout,
            last ? perm : nullptr, col, src, weight_csr, edge_weight);
        PYG_LAUNCH_CHECK();
        kin = kout;
        vin = vout;
        shift += bits;
    }
    return PYG_OK;
}

extern "C" int pyg_validate_coo(const int64_t *edge_index, int64_t E, int64_t N, int64_t *bad_count, void *stream) {
    if (E < 0 || N < 0 || !bad_count || (E > 0 && !edge_index)) return PYG_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    PYG_TRY(fill<int64_t>(bad_count, 1, 0, s));
    if (E == 0) return PYG_OK;
    k_validate_coo<<<grid_for(2 * E, kBlock * 8, 4096), kBlock, 0, s>>>(edge_index, 2 * E, N,
                                                                          reinterpret_cast<unsigned long long *>(bad_count));
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

extern "C" int pyg_validate_batch(const int64_t *batch, int64_t N, int64_t B, int64_t *bad_count, void *stream) {
    if (N < 0 || B < 0 || !bad_count || (N > 0 && !batch)) return PYG_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    PYG_TRY(fill<int64_t>(bad_count, 1, 0, s));
    if (N == 0) return PYG_OK;
    k_validate_batch<<<grid_for(N, kBlock * 8, 4096), kBlock, 0, s>>>(batch, N, B, reinterpret_cast<unsigned long long *>(bad_count));
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}
