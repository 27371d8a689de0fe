// Preprocessing: in-degree, stable COO -> target-sorted CSR, index validation.
// (The radix payload is packed into one 64-bit word per edge when the ids fit;
// see "packed sort" below.)
//
// The CSR is the row-ordered ("coalesced") layout that Appendix A says a
// sparse-matrix product needs and that should be built once, as
// preprocessing. It is built here with a stable LSD radix sort of the target
// ids that carries (edge id, source, weight) as payload, so no pass gathers
// at random:
//   per pass  k_radix_hist     digit counts per tile, digit-major
//             device scan      -> global offset of every (digit, tile)
//             k_radix_scatter  each wavefront ranks its 1024 keys against
//                              wave-private LDS counters (ballot match on
//                              the digit bits), the tile combines the four
//                              waves in order, stages a tile-local
//                              permutation in LDS and writes every digit run
//                              contiguously.
//   then      k_row_bounds     rowptr from the key changes of the sorted keys
//                              (k_row_bounds_low when the packed sort kept
//                              only each key's bits below its last digit).
// Elements keep their order inside equal digits in every pass, so the slots
// of a row end in ascending COO edge id and the result is unique. The same
// packed passes also partition (edge id, slot) pairs for the LDS-blocked
// inverse permutation of the transpose map (inverse_perm_sorted).
//
// In-degree counting uses LDS-privatised histograms over slices of the node
// range (no global atomics on the edge stream): every workgroup counts the
// targets of one edge partition that fall into its slice, then writes its
// counters once; a reduce pass sums the partitions in a fixed order. (One
// 32-bit global atomic per edge instead measured 4.8 ms against 0.93 ms on
// the large power-law graph.)
#include "common.hpp"

namespace pyg {
namespace {

#ifndef PYG_RADIX_ITEMS
#define PYG_RADIX_ITEMS 8  // 2048-key tiles: twice the workgroups of 16, measured faster with XCD-major tiles
#endif
#ifndef PYG_RADIX_BITS
#define PYG_RADIX_BITS 7  // 18-bit ids: three 6-bit passes, whose 64-key runs write whole lines
#endif
constexpr int kItems = PYG_RADIX_ITEMS;                     // keys per thread per tile
#ifndef PYG_SORT_THREADS
#define PYG_SORT_THREADS 256
#endif
constexpr int kSortBlock = PYG_SORT_THREADS;                // threads per tile of the radix kernels
constexpr int kWaveKeys = kWave * kItems;                   // keys ranked by one wavefront
constexpr int64_t kTile = (int64_t)kSortBlock * kItems;     // keys per tile
constexpr int kMaxDigitBits = PYG_RADIX_BITS;               // widest digit of one pass
static_assert(kTile <= 65536, "tile-local indices are staged as 16-bit");
constexpr int kMaxRadix = 1 << kMaxDigitBits;
constexpr int kWaves = kSortBlock / kWave;

// ------------------------------------------------------------------ degree

// Count targets of one edge partition that fall in one node slice; write
// the slice's counters to partial[partition][node]. One workgroup of 1024
// threads holds a whole slice in LDS, so each thread keeps 8 target loads in
// flight. Every slice reads the whole partition: the workgroup -> (slice,
// partition) map puts the slices of a partition on one XCD (workgroups are
// dealt to the 8 XCDs in turn), so that one XCD's L2 serves the re-reads.
constexpr int kHistThreads = 1024;
constexpr int kHistUnroll = 8;

__global__ __launch_bounds__(kHistThreads) void k_hist_slice(const int64_t *__restrict__ dst, int64_t E, int64_t N,
                                                             int64_t slice, int64_t nslices, int64_t part_len,
                                                             uint32_t *__restrict__ partial) {
    extern __shared__ uint32_t cnt[];
    const int64_t L = xcd_major(blockIdx.x, gridDim.x);
    const int64_t sl = L % nslices, part = L / nslices;
    const int64_t n0 = sl * slice;
    const int64_t n1 = (n0 + slice) < N ? (n0 + slice) : N;
    const int64_t len = n1 - n0;
    for (int64_t i = threadIdx.x; i < len; i += kHistThreads) cnt[i] = 0;
    __syncthreads();
    const int64_t e0 = part * part_len;
    const int64_t e1 = (e0 + part_len) < E ? (e0 + part_len) : E;
    int64_t k = e0 + threadIdx.x;
    for (; k + (kHistUnroll - 1) * kHistThreads < e1; k += kHistUnroll * kHistThreads) {
        int64_t d[kHistUnroll];
#pragma unroll
        for (int u = 0; u < kHistUnroll; ++u) d[u] = dst[k + u * kHistThreads] - n0;
#pragma unroll
        for (int u = 0; u < kHistUnroll; ++u)
            if (static_cast<uint64_t>(d[u]) < static_cast<uint64_t>(len)) atomicAdd(&cnt[d[u]], 1u);
    }
    for (; k < e1; k += kHistThreads) {
        const int64_t d = dst[k] - n0;
        if (static_cast<uint64_t>(d) < static_cast<uint64_t>(len)) atomicAdd(&cnt[d], 1u);
    }
    __syncthreads();
    uint32_t *out = partial + part * N + n0;
    for (int64_t i = threadIdx.x; i < len; i += kHistThreads) out[i] = cnt[i];
}

// deg[i] = sum over partitions of partial[p][i] (fixed order).
template <typename Out>
__global__ void k_hist_reduce(const uint32_t *__restrict__ partial, int64_t N, int64_t parts, Out *__restrict__ out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x) {
        uint64_t s = 0;
        for (int64_t p = 0; p < parts; ++p) s += partial[p * N + i];
        out[i] = static_cast<Out>(s);
    }
}

struct HistPlan {
    int64_t slice, nslices, parts, part_len;
    size_t lds;
};

HistPlan hist_plan(int64_t E, int64_t N) {
    static const int lds_limit = [] {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
            v = 64 * 1024;
        return v < 160 * 1024 ? v : 160 * 1024;
    }();
    HistPlan h{};
    h.slice = (lds_limit - 1024) / 4;
    if (h.slice > N) h.slice = N > 0 ? N : 1;
    h.nslices = (N + h.slice - 1) / h.slice;
    if (h.nslices < 1) h.nslices = 1;
    // about 1024 workgroups in total, each partition at least 64K edges
    int64_t parts = 1024 / h.nslices;
    const int64_t by_size = (E + 65535) / 65536;
    if (parts > by_size) parts = by_size;
    if (parts < 1) parts = 1;
    h.part_len = (E + parts - 1) / parts;
    h.parts = h.part_len > 0 ? (E + h.part_len - 1) / h.part_len : 1;
    h.lds = static_cast<size_t>(h.slice) * 4;
    return h;
}

size_t hist_workspace(int64_t E, int64_t N) {
    const HistPlan h = hist_plan(E, N);
    return align_up(static_cast<size_t>(h.parts) * N * 4, 256) + 256;
}

template <typename Out>
int count_targets(const int64_t *dst, int64_t E, int64_t N, Out *out, void *ws, hipStream_t s) {
    if (N == 0) return PYG_OK;
    if (E == 0) return fill<Out>(out, N, Out(0), s);
    const HistPlan h = hist_plan(E, N);
    uint32_t *partial = static_cast<uint32_t *>(ws);
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(k_hist_slice), hipFuncAttributeMaxDynamicSharedMemorySize,
                            static_cast<int>(h.lds)) != hipSuccess)
        return PYG_ERR_HIP;
    k_hist_slice<<<(unsigned)(h.nslices * h.parts), kHistThreads, h.lds, s>>>(dst, E, N, h.slice, h.nslices, h.part_len,
                                                                              partial);
    PYG_LAUNCH_CHECK();
    k_hist_reduce<Out><<<grid_for(N, kBlock), kBlock, 0, s>>>(partial, N, h.parts, out);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

// ------------------------------------------------------------- radix sort

// The sort key of an edge: its target, or for a source-blocked CSR
// (bsize > 0) the source block above the target's bits,
// (source / bsize) << tb | target, so that the sorted order is by source
// block, then target, then edge id. The low digits then depend on the
// target alone (the first pass reads no source ids); the sorted keys are
// turned into virtual rows (source block) * N + target at the end.
struct SortKey {
    int64_t bsize;   // 0: plain CSR
    int64_t N;
    int tb;          // bits of a target id
    uint64_t bmagic; // source / bsize = (source * bmagic) >> bshift for sources below 2^31
    int bshift;
};

__device__ __forceinline__ uint32_t first_key(const int64_t *__restrict__ dst64, const int64_t *__restrict__ src64,
                                              int64_t i, SortKey sk, bool with_block = true) {
    const uint32_t t = static_cast<uint32_t>(dst64[i]);
    if (sk.bsize == 0 || !with_block) return t;
    const uint32_t b = static_cast<uint32_t>((static_cast<uint64_t>(static_cast<uint32_t>(src64[i])) * sk.bmagic) >>
                                             sk.bshift);
    return (b << sk.tb) | t;
}

// A sorted key as the row of the CSR it was sorted into.
__device__ __forceinline__ uint32_t key_row(uint32_t k, SortKey sk) {
    if (sk.bsize == 0) return k;
    return (k >> sk.tb) * static_cast<uint32_t>(sk.N) + (k & ((1u << sk.tb) - 1u));
}

struct Payload {  // one sort buffer: key plus carried fields
    uint32_t *key;
    uint32_t *id;
    uint32_t *src;
    float *w;
};

__global__ __launch_bounds__(kSortBlock) void k_radix_hist(const int64_t *__restrict__ dst64, const int64_t *__restrict__ src64,
                                                       const uint32_t *__restrict__ keys, SortKey sk,
                                                       int64_t E, int shift, int bits, int64_t ntiles,
                                                       uint32_t *__restrict__ hist) {
    __shared__ uint32_t h[kMaxRadix];
    const int radix = 1 << bits;
    const uint32_t mask = radix - 1;
    for (int i = threadIdx.x; i < radix; i += kSortBlock) h[i] = 0;
    __syncthreads();
    const int64_t tile = blockIdx.x;
    const int64_t base = tile * kTile + threadIdx.x;
#pragma unroll 4
    for (int r = 0; r < kItems; ++r) {
        const int64_t i = base + (int64_t)r * kSortBlock;
        if (i < E) {
            const uint32_t key = dst64 ? first_key(dst64, src64, i, sk, shift + bits > sk.tb) : keys[i];
            atomicAdd(&h[(key >> shift) & mask], 1u);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < radix; i += kSortBlock) hist[(int64_t)i * ntiles + tile] = h[i];
}

// Stable rank of one tile's elements by digit. dig[r] is the digit of the
// wave's element r (0xFFFFFFFF past the end); on return slot[r] is its
// position in the tile sorted by digit (equal digits keep tile order),
// start[d] the first sorted position of digit d and gbase[d] the global slot
// of sorted position 0 of digit d's run (so sorted position j of digit d
// goes to gbase[d] + j). Each wavefront ranks its 1024 elements with ballot
// matches on the digit bits against wave-private LDS counters; the tile then
// combines the four waves in order.
template <int MAXR>
__device__ __forceinline__ void rank_tile(const uint32_t (&dig)[kItems], uint32_t (&slot)[kItems],
                                          uint32_t (&wcnt)[kWaves][MAXR], uint32_t (&start)[MAXR],
                                          int64_t (&gbase)[MAXR], const uint32_t *__restrict__ offsets,
                                          int64_t ntiles, int64_t tile, int bits) {
    const int radix = 1 << bits;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    for (int i = lane; i < radix; i += kWave) wcnt[wave][i] = 0;
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const bool valid = dig[r] != 0xFFFFFFFFu;
        const uint32_t d = valid ? dig[r] : 0u;
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < bits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        const uint32_t before = __popcll(peers & lt_mask);
        const uint32_t base = valid ? wcnt[wave][d] : 0u;
        __builtin_amdgcn_wave_barrier();
        if (valid && before == 0) wcnt[wave][d] = base + __popcll(peers);
        __builtin_amdgcn_wave_barrier();
        slot[r] = base + before;
    }
    __syncthreads();

    // per digit, prefix over waves; then the tile start of each digit run
    for (int t = threadIdx.x; t < radix; t += kSortBlock) {
        uint32_t acc = 0;
#pragma unroll
        for (int wv = 0; wv < kWaves; ++wv) {
            const uint32_t c = wcnt[wv][t];
            wcnt[wv][t] = acc;
            acc += c;
        }
        start[t] = acc;  // digit total, scanned below
    }
    __syncthreads();
    if (threadIdx.x < kWave) {
        // one wave scans the digit totals: a few per lane, then a lane prefix
        constexpr int per = (MAXR + kWave - 1) / kWave;
        uint32_t v[per];
        uint32_t sum = 0;
#pragma unroll
        for (int j = 0; j < per; ++j) {
            const int t = lane * per + j;
            v[j] = t < radix ? start[t] : 0u;
            sum += v[j];
        }
        uint32_t incl = sum;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const uint32_t y = __shfl_up(incl, d, kWave);
            if (lane >= d) incl += y;
        }
        uint32_t run = incl - sum;
#pragma unroll
        for (int j = 0; j < per; ++j) {
            const int t = lane * per + j;
            if (t < radix) start[t] = run;
            run += v[j];
        }
    }
    __syncthreads();
    for (int t = threadIdx.x; t < radix; t += kSortBlock)
        gbase[t] = (int64_t)offsets[(int64_t)t * ntiles + tile] - (int64_t)start[t];
#pragma unroll
    for (int r = 0; r < kItems; ++r)
        if (dig[r] != 0xFFFFFFFFu) slot[r] += start[dig[r]] + wcnt[wave][dig[r]];
}

// One stable scatter pass. Tile element order: wave w owns elements
// [w*1024, (w+1)*1024) of the tile, visited 64 at a time in lane order.
// Every global read is coalesced: each field (key, edge id, source, weight)
// is loaded in tile order, scattered into LDS in sorted order, and written
// out run by run, so no pass gathers from global memory.
__global__ __launch_bounds__(kSortBlock) void k_radix_scatter(
    const int64_t *__restrict__ dst64, const int64_t *__restrict__ src64, const float *__restrict__ w_in,
    Payload in, Payload out, int64_t *__restrict__ perm, int32_t *__restrict__ col, float *__restrict__ wcsr,
    int64_t E, int shift, int bits, int64_t ntiles, const uint32_t *__restrict__ offsets, int last, SortKey sk) {
    __shared__ uint32_t wcnt[kWaves][kMaxRadix];  // per-wave running counts, then per-wave prefixes
    __shared__ uint32_t start[kMaxRadix];         // first staged slot of each digit in the tile
    __shared__ int64_t gbase[kMaxRadix];          // global slot of staged slot 0 of each digit run
    __shared__ uint32_t stage[kTile];             // one field of the tile, in sorted order
    __shared__ uint16_t sdig[kTile];              // digit of each sorted slot
    const uint32_t mask = (1u << bits) - 1;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t tile = xcd_major(blockIdx.x, gridDim.x);  // neighbouring tiles write neighbouring runs
    const int64_t tbase = tile * kTile;
    const int64_t tlen = (E - tbase) < kTile ? (E - tbase) : kTile;
    const int64_t ebase = tbase + wave * kWaveKeys + lane;  // element of round r: ebase + r * 64

    // phase A: load this wave's keys
    uint32_t key[kItems], dig[kItems], slot[kItems];
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const int64_t i = ebase + r * kWave;
        key[r] = (i < E) ? (dst64 ? first_key(dst64, src64, i, sk) : in.key[i]) : 0u;
        dig[r] = (i < E) ? (key[r] >> shift) & mask : 0xFFFFFFFFu;
    }
    rank_tile<kMaxRadix>(dig, slot, wcnt, start, gbase, offsets, ntiles, tile, bits);

    // field 0: the key (and the digit of every sorted slot)
#pragma unroll
    for (int r = 0; r < kItems; ++r)
        if (dig[r] != 0xFFFFFFFFu && slot[r] < kTile) {
            stage[slot[r]] = key[r];
            sdig[slot[r]] = static_cast<uint16_t>(dig[r]);
        }
    __syncthreads();
    uint32_t *key_out = out.key;
    for (int64_t j = threadIdx.x; j < tlen; j += kSortBlock) {
        const int64_t pos = gbase[sdig[j]] + j;
        if (pos >= 0 && pos < E) key_out[pos] = last ? key_row(stage[j], sk) : stage[j];  // bounds hold for a consistent ranking
    }

    // fields 1..3: edge id, source, weight
    for (int fld = 1; fld <= 3; ++fld) {
        if (fld == 3 && !(dst64 ? w_in : in.w)) break;
        __syncthreads();  // stage[] free again
        uint32_t v[kItems];
#pragma unroll
        for (int r = 0; r < kItems; ++r) {
            const int64_t i = ebase + r * kWave;
            uint32_t x = 0;
            if (i < E) {
                if (fld == 1) x = dst64 ? static_cast<uint32_t>(i) : in.id[i];
                else if (fld == 2) x = dst64 ? static_cast<uint32_t>(src64[i]) : in.src[i];
                else x = dst64 ? __float_as_uint(w_in[i]) : __float_as_uint(in.w[i]);
            }
            v[r] = x;
        }
#pragma unroll
        for (int r = 0; r < kItems; ++r)
            if (dig[r] != 0xFFFFFFFFu && slot[r] < kTile) stage[slot[r]] = v[r];
        __syncthreads();
        for (int64_t j = threadIdx.x; j < tlen; j += kSortBlock) {
            const int64_t pos = gbase[sdig[j]] + j;
            if (pos < 0 || pos >= E) continue;
            const uint32_t x = stage[j];
            if (last) {
                if (fld == 1) {
                    if (perm) perm[pos] = x;
                }
                else if (fld == 2) col[pos] = static_cast<int32_t>(x);
                else if (wcsr) wcsr[pos] = __uint_as_float(x);
            } else {
                if (fld == 1) out.id[pos] = x;
                else if (fld == 2) out.src[pos] = x;
                else out.w[pos] = __uint_as_float(x);
            }
        }
    }
}

// ------------------------------------------------------------ packed sort
// When kb + nb + ib <= 64 (kb bits of the sort key, nb of a node id, ib of an
// edge id), an element travels as one 64-bit word  key << (nb + ib) | source << ib | id:
// 8 bytes per element and pass instead of 12 (the large power-law graph:
// 3.63 -> 3.00 ms). Digits stay at most 7 bits (three 6-bit passes for 18-bit
// ids): two 9-bit passes measured slower (3.71 ms), their 8-element runs per
// tile write partial lines; so did two passes of 10 and 9 bits with 2-byte
// digits, 2048- or 4096-element tiles (3.2-4.0 ms against 2.1 ms).
#ifndef PYG_RADIX_BITS_PACKED
#define PYG_RADIX_BITS_PACKED 7
#endif
constexpr int kMaxDigitBitsP = PYG_RADIX_BITS_PACKED;
constexpr int kMaxRadixP = 1 << kMaxDigitBitsP;
// the scatter hands the next pass its digits as one byte per element
static_assert(kMaxDigitBitsP <= 8, "packed-sort digits are stored in one byte");

struct Packing {
    int kb;  // bits of the sort key (the target, or the virtual row of a blocked CSR)
    int nb;  // bits of a node id (0: no node id field)
    int ib;  // bits of an edge id
    SortKey sk;
};

__device__ __forceinline__ uint64_t pack_edge(const int64_t *__restrict__ dst64, const int64_t *__restrict__ src64,
                                              int64_t i, Packing pk) {
    return (static_cast<uint64_t>(first_key(dst64, src64, i, pk.sk)) << (pk.nb + pk.ib)) |
           (pk.nb ? static_cast<uint64_t>(src64[i]) << pk.ib : 0ull) | static_cast<uint64_t>(i);
}

// Digit counts per tile (digit-major) of the packed elements; pass 0 packs
// from the COO itself, later passes read the one-byte digits the previous
// scatter wrote. One workgroup counts TPW neighbouring tiles into LDS
// counters of its own per tile (K copies of each, lane % K picking one, so
// that lanes of a skewed digit spread their LDS atomics) and writes them as
// TPW neighbouring words per digit; the byte digits arrive 16 to a load.
// (One workgroup per 2048-element tile spent 145 us on the 115 MB of digits
// of the large power-law graph: launch and flush overhead, 4-byte scattered
// writes.)
constexpr int kHistTiles0 = 1;  // tiles per workgroup, pass 0 (reads the COO: 8 measured no faster)
static_assert(kItems % 2 == 0, "pass 0 reads its 8-byte ids in pairs");
constexpr int kHistTiles = 8;   // tiles per workgroup, later passes (read byte digits)
constexpr int kHistCopies = 4;  // counter copies (8 measured no faster, 1 slower on the skewed top digit)
static_assert(kTile % 16 == 0, "a 16-byte digit load stays in one tile");

template <int TPW, int K>
__global__ __launch_bounds__(kSortBlock) void k_radix_hist64(const int64_t *__restrict__ dst64,
                                                         const int64_t *__restrict__ src64,
                                                         const uint64_t *__restrict__ keys,
                                                         const uint8_t *__restrict__ dig8, int64_t E, int shift,
                                                         int bits, int64_t ntiles, Packing pk,
                                                         uint32_t *__restrict__ hist) {
    // 16-byte digit loads per thread, when a workgroup's digits split into whole loads
    constexpr bool kVecOk = (TPW * kTile) % (16 * kSortBlock) == 0;
    constexpr int kVec = kVecOk ? (int)(TPW * kTile / 16 / kSortBlock) : 1;
    __shared__ uint32_t h[TPW * kMaxRadixP * K];  // [tile][digit][copy]
    const int radix = 1 << bits;
    const uint32_t mask = radix - 1;
    const int copy = K > 1 ? (int)(threadIdx.x % K) : 0;
    for (int i = threadIdx.x; i < TPW * kMaxRadixP * K; i += kSortBlock) h[i] = 0;
    __syncthreads();
    const int64_t t0 = (int64_t)blockIdx.x * TPW;
    const int64_t base = t0 * kTile;
    const int64_t span = (E - base) < TPW * kTile ? (E - base) : TPW * kTile;  // elements here
    if (kVecOk && dig8 && (reinterpret_cast<uintptr_t>(dig8) & 15) == 0) {
        uint4 q[kVec];
#pragma unroll
        for (int r = 0; r < kVec; ++r) {
            const int64_t o = (int64_t)(r * kSortBlock + threadIdx.x) * 16;
            q[r] = (o + 16 <= span) ? *reinterpret_cast<const uint4 *>(dig8 + base + o) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int r = 0; r < kVec; ++r) {
            const int64_t o = (int64_t)(r * kSortBlock + threadIdx.x) * 16;
            uint32_t *hh = h + (o / kTile) * kMaxRadixP * K + copy;
            if (o + 16 <= span) {
                const uint32_t w4[4] = {q[r].x, q[r].y, q[r].z, q[r].w};
#pragma unroll
                for (int k = 0; k < 16; ++k) atomicAdd(&hh[((w4[k >> 2] >> (8 * (k & 3))) & mask) * K], 1u);
            } else {
                for (int64_t k = o; k < span; ++k) atomicAdd(&hh[(dig8[base + k] & mask) * K], 1u);
            }
        }
    } else if (TPW == 1 && dst64 && !(shift + bits > pk.sk.tb && pk.sk.bsize)) {
        // pass 0 over the targets: pairs of 8-byte ids per 16-byte load, from
        // the first 16-byte boundary (a leading odd element and a trailing
        // single one taken alone)
        const int64_t *d = dst64 + base;
        const int a = (reinterpret_cast<uintptr_t>(d) & 15) ? 1 : 0;
        const int64_t npair = (span - a) >> 1;
        uint32_t *hh = h + copy;
        constexpr int kP = kItems / 2;  // pairs per thread
        longlong2 q[kP];
#pragma unroll
        for (int r = 0; r < kP; ++r) {
            const int64_t j = (int64_t)r * kSortBlock + threadIdx.x;
            q[r] = j < npair ? *reinterpret_cast<const longlong2 *>(d + a + 2 * j) : make_longlong2(0, 0);
        }
#pragma unroll
        for (int r = 0; r < kP; ++r) {
            const int64_t j = (int64_t)r * kSortBlock + threadIdx.x;
            if (j < npair) {
                atomicAdd(&hh[((static_cast<uint32_t>(q[r].x) >> shift) & mask) * K], 1u);
                atomicAdd(&hh[((static_cast<uint32_t>(q[r].y) >> shift) & mask) * K], 1u);
            }
        }
        if (threadIdx.x == 0 && a) atomicAdd(&hh[((static_cast<uint32_t>(d[0]) >> shift) & mask) * K], 1u);
        if (threadIdx.x == 1 && ((span - a) & 1)) atomicAdd(&hh[((static_cast<uint32_t>(d[span - 1]) >> shift) & mask) * K], 1u);
    } else {
        for (int64_t j0 = 0; j0 < span; j0 += (int64_t)kSortBlock * kItems) {
            uint32_t d[kItems];
#pragma unroll
            for (int r = 0; r < kItems; ++r) {
                const int64_t j = j0 + (int64_t)r * kSortBlock + threadIdx.x;
                const int64_t i = base + j;
                d[r] = j >= span ? 0xFFFFFFFFu
                       : dig8 ? dig8[i]
                       : dst64 ? static_cast<uint32_t>(
                                     first_key(dst64, src64, i, pk.sk, shift + bits > pk.sk.tb) >> shift)
                               : static_cast<uint32_t>(keys[i] >> (pk.nb + pk.ib + shift));
            }
            uint32_t *hh = h + (j0 / kTile) * kMaxRadixP * K + copy;
#pragma unroll
            for (int r = 0; r < kItems; ++r)
                if (d[r] != 0xFFFFFFFFu) atomicAdd(&hh[(d[r] & mask) * K], 1u);
        }
    }
    __syncthreads();
    const int nt = (ntiles - t0) < TPW ? (int)(ntiles - t0) : TPW;
    for (int k = threadIdx.x; k < radix * TPW; k += kSortBlock) {
        const int d = k / TPW, tt = k % TPW;
        if (tt >= nt) continue;
        uint32_t c = 0;
#pragma unroll
        for (int cp = 0; cp < K; ++cp) c += h[(tt * kMaxRadixP + d) * K + cp];
        hist[(int64_t)d * ntiles + t0 + tt] = c;
    }
}

// One stable scatter pass over packed elements (same tile order and ranking
// as k_radix_scatter). The last pass (last != 0) unpacks into perm, col and
// the sorted keys: as rows (last = 1), or (last = 2) as the key bits below
// this pass's digit, 2 bytes each, when there are at most 16 of them (the
// digit itself is known from the digit offsets; k_row_bounds_low).
__global__ __launch_bounds__(kSortBlock) void k_radix_scatter64(
    const int64_t *__restrict__ dst64, const int64_t *__restrict__ src64, const float *__restrict__ w_in,
    const uint64_t *__restrict__ in, const float *__restrict__ in_w, uint64_t *__restrict__ out,
    float *__restrict__ out_w, int64_t *__restrict__ perm, int32_t *__restrict__ col, float *__restrict__ wcsr,
    uint32_t *__restrict__ sorted_key, int64_t E, int shift, int bits, int64_t ntiles,
    const uint32_t *__restrict__ offsets, int last, Packing pk, uint8_t *__restrict__ next_dig, int next_shift,
    int next_bits) {
    __shared__ uint32_t wcnt[kWaves][kMaxRadixP];
    __shared__ uint32_t start[kMaxRadixP];
    __shared__ int64_t gbase[kMaxRadixP];
    __shared__ uint64_t stage[kTile];  // the tile's elements in sorted order
    __shared__ uint16_t sdig[kTile];
    const uint64_t mask = (1ull << bits) - 1;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t tile = xcd_major(blockIdx.x, gridDim.x);  // neighbouring tiles write neighbouring runs
    const int64_t tbase = tile * kTile;
    const int64_t tlen = (E - tbase) < kTile ? (E - tbase) : kTile;
    const int64_t ebase = tbase + wave * kWaveKeys + lane;
    const int koff = pk.nb + pk.ib;

    uint64_t el[kItems];
    uint32_t dig[kItems], slot[kItems];
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const int64_t i = ebase + r * kWave;
        el[r] = (i < E) ? (dst64 ? pack_edge(dst64, src64, i, pk) : in[i]) : 0ull;
        dig[r] = (i < E) ? static_cast<uint32_t>((el[r] >> (koff + shift)) & mask) : 0xFFFFFFFFu;
    }
    rank_tile<kMaxRadixP>(dig, slot, wcnt, start, gbase, offsets, ntiles, tile, bits);
#pragma unroll
    for (int r = 0; r < kItems; ++r)
        if (dig[r] != 0xFFFFFFFFu && slot[r] < kTile) {
            stage[slot[r]] = el[r];
            sdig[slot[r]] = static_cast<uint16_t>(dig[r]);
        }
    __syncthreads();
    const uint64_t idmask = (1ull << pk.ib) - 1, nodemask = (1ull << pk.nb) - 1;
    for (int64_t j = threadIdx.x; j < tlen; j += kSortBlock) {
        const int64_t pos = gbase[sdig[j]] + j;
        if (pos < 0 || pos >= E) continue;  // bounds hold for a consistent ranking
        const uint64_t e = stage[j];
        if (last) {
            if (perm) perm[pos] = static_cast<int64_t>(e & idmask);
            col[pos] = static_cast<int32_t>((e >> pk.ib) & nodemask);
            if (last == 2)
                reinterpret_cast<uint16_t *>(sorted_key)[pos] =
                    static_cast<uint16_t>((e >> koff) & ((1ull << shift) - 1));
            else
                sorted_key[pos] = key_row(static_cast<uint32_t>(e >> koff), pk.sk);
        } else {
            out[pos] = e;
            // the next pass's digit, one byte: its histogram reads these instead of the 8-byte words
            if (next_dig) next_dig[pos] = static_cast<uint8_t>((e >> (koff + next_shift)) & ((1u << next_bits) - 1));
        }
    }
    // the weight, if any, as a second staged field
    if (!(dst64 ? w_in : in_w)) return;
    __syncthreads();
    uint32_t *stage32 = reinterpret_cast<uint32_t *>(stage);
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const int64_t i = ebase + r * kWave;
        if (dig[r] != 0xFFFFFFFFu && slot[r] < kTile)
            stage32[slot[r]] = __float_as_uint(dst64 ? w_in[i] : in_w[i]);
    }
    __syncthreads();
    for (int64_t j = threadIdx.x; j < tlen; j += kSortBlock) {
        const int64_t pos = gbase[sdig[j]] + j;
        if (pos < 0 || pos >= E) continue;
        const float w = __uint_as_float(stage32[j]);
        if (last) {
            if (wcsr) wcsr[pos] = w;
        } else {
            out_w[pos] = w;
        }
    }
}

// rowptr from the sorted target ids: slot p starts every row in (key[p-1], key[p]]
// (key[-1] = -1, key[E] = N; slot E closes the trailing rows, rowptr[N] = E).
// Each thread owns 8 consecutive slots, read as two 16-byte loads.
__global__ void k_row_bounds(const uint32_t *__restrict__ key, int64_t E, int64_t N, int64_t *__restrict__ rowptr) {
    // N: the number of rows (target ids, or virtual rows of a blocked CSR)
    constexpr int S = 8;  // slots per thread: two 16-byte loads
    const int64_t p0 = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * S;
    if (p0 > E) return;
    int64_t k[S + 1];
    k[0] = p0 == 0 ? -1 : static_cast<int64_t>(key[p0 - 1]);
    if (p0 + S <= E) {
        const uint4 a = *reinterpret_cast<const uint4 *>(key + p0);
        const uint4 b = *reinterpret_cast<const uint4 *>(key + p0 + 4);
        k[1] = a.x, k[2] = a.y, k[3] = a.z, k[4] = a.w, k[5] = b.x, k[6] = b.y, k[7] = b.z, k[8] = b.w;
    } else {
#pragma unroll
        for (int i = 0; i < S; ++i) k[i + 1] = p0 + i < E ? static_cast<int64_t>(key[p0 + i]) : N;
    }
#pragma unroll
    for (int i = 0; i <= S; ++i) k[i] = k[i] > N ? N : k[i];
#pragma unroll
    for (int i = 0; i < S; ++i) {
        const int64_t p = p0 + i;
        if (p > E) break;
        for (int64_t r = k[i] + 1; r <= k[i + 1]; ++r) rowptr[r] = p;
    }
}

// The start of every digit of the sort's last pass (the exclusive scan of
// its digit-major counts at tile 0), and E after the last digit.
__global__ void k_digit_starts(const uint32_t *__restrict__ scanned, int64_t ntiles, int radix, int64_t E,
                               uint32_t *__restrict__ dstart) {
    for (int t = threadIdx.x; t <= radix; t += blockDim.x)
        dstart[t] = t < radix ? scanned[(int64_t)t * ntiles] : static_cast<uint32_t>(E);
}

// k_row_bounds over keys stored as their bits below the last pass's digit
// (L of them, 2 bytes per slot): the key of slot p is d << L | low[p] with d
// the digit whose range [dstart[d], dstart[d+1]) holds p. 16 slots per thread
// (8 measured 104 against 79 us on the large power-law graph: the digit
// search and the LDS copy of the digit starts are per thread and workgroup).
constexpr int kRowBoundsLowSlots = 16;
__global__ __launch_bounds__(kBlock) void k_row_bounds_low(const uint16_t *__restrict__ low,
                                                           const uint32_t *__restrict__ dstart_g, int radix, int L,
                                                           SortKey sk, int64_t E, int64_t N,
                                                           int64_t *__restrict__ rowptr) {
    constexpr int S = kRowBoundsLowSlots;  // slots per thread: two 16-byte loads
    __shared__ uint32_t dstart[kMaxRadixP + 1];
    for (int t = threadIdx.x; t <= radix; t += blockDim.x) dstart[t] = dstart_g[t];
    __syncthreads();
    const int64_t p0 = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) * S;
    if (p0 > E) return;
    // the digit of slot max(p0 - 1, 0): the last d with dstart[d] <= p
    const int64_t q = p0 > 0 ? p0 - 1 : 0;
    int lo = 0, hi = radix - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (static_cast<int64_t>(dstart[mid]) <= q) lo = mid;
        else hi = mid - 1;
    }
    int d = lo;
    int64_t next = d + 1 < radix ? static_cast<int64_t>(dstart[d + 1]) : INT64_MAX;  // where digit d ends
    auto row_of = [&](int64_t p, uint32_t lw) -> int64_t {
        while (p >= next) {
            ++d;
            next = d + 1 < radix ? static_cast<int64_t>(dstart[d + 1]) : INT64_MAX;
        }
        return static_cast<int64_t>(key_row((static_cast<uint32_t>(d) << L) | lw, sk));
    };
    int64_t k[S + 1];
    k[0] = p0 == 0 ? -1 : row_of(p0 - 1, low[p0 - 1]);
    if (p0 + S <= E) {
        uint32_t w[S / 2];
#pragma unroll
        for (int v = 0; v < S / 8; ++v) {
            const uint4 a = *reinterpret_cast<const uint4 *>(low + p0 + 8 * v);
            w[4 * v] = a.x, w[4 * v + 1] = a.y, w[4 * v + 2] = a.z, w[4 * v + 3] = a.w;
        }
#pragma unroll
        for (int i = 0; i < S; ++i) k[i + 1] = row_of(p0 + i, (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
    } else {
        for (int i = 0; i < S; ++i) k[i + 1] = p0 + i < E ? row_of(p0 + i, low[p0 + i]) : N;
    }
#pragma unroll
    for (int i = 0; i <= S; ++i) k[i] = k[i] > N ? N : k[i];
#pragma unroll
    for (int i = 0; i < S; ++i) {
        const int64_t p = p0 + i;
        if (p > E) break;
        for (int64_t r = k[i] + 1; r <= k[i + 1]; ++r) rowptr[r] = p;
    }
}

__global__ void k_gather_edges(const int64_t *__restrict__ perm, int64_t E, const float *__restrict__ in,
                               float *__restrict__ out) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < E; p += (int64_t)gridDim.x * blockDim.x)
        out[p] = in[perm[p]];
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

// Digit plan for keys of b bits: passes and bits per pass (at least one pass).
void digit_plan(int b, int *nb, int *passes, int *bpp) {
    *nb = b;
    *passes = (b + kMaxDigitBits - 1) / kMaxDigitBits;
    *bpp = (b + *passes - 1) / *passes;
}

// Source blocks: B blocks of ceil(N / B) consecutive source ids (B = 1: the
// plain CSR, keyed by target alone). The block of a source is a division by
// the invariant bsize, done as a multiply and shift (Granlund and
// Montgomery, division by invariant integers using multiplication, 1994):
// with l = ceil(log2 bsize) and m = floor(2^(31+l) / bsize) + 1, floor(n /
// bsize) = floor(n m / 2^(31+l)) for every 0 <= n < 2^31, and n m < 2^64
// (m < 2^33). The GPU has no integer divide instruction: a division by a
// runtime value is a reciprocal-and-correction sequence per edge.
SortKey sort_key(int64_t N, int64_t B) {
    SortKey sk{};
    sk.bsize = B > 1 ? (N + B - 1) / B : 0;
    sk.N = N;
    sk.tb = 1;
    while (sk.tb < 31 && (int64_t(1) << sk.tb) < N) ++sk.tb;
    if (sk.bsize > 0) {
        int l = 0;
        while ((int64_t(1) << l) < sk.bsize) ++l;
        sk.bmagic = ((uint64_t(1) << (31 + l)) / static_cast<uint64_t>(sk.bsize)) + 1;
        sk.bshift = 31 + l;
    }
    return sk;
}

// Bits of the sort key for B source blocks (B = 1: the target alone).
int key_bits(int64_t N, int64_t B) {
    const SortKey sk = sort_key(N, B);
    if (B <= 1) return sk.tb;
    int bb = 0;
    while ((int64_t(1) << bb) < B) ++bb;
    return sk.tb + bb;
}

// Digit bits of packed pass p when kb key bits are spread over `passes`
// passes: as even as possible, the wider digits last (19-bit keys as 6, 6, 7:
// a 6-bit digit's 32-element runs write whole lines; 7, 7, 5 measured 0.1 ms
// slower on the large power-law graph).
int pass_bits(int kb, int passes, int p) {
    const int base = kb / passes, extra = kb % passes;
    return base + (p >= passes - extra ? 1 : 0);
}

// Packed layout when a sort key, a node id and an edge id fit 64 bits.
bool packed_plan(int64_t E, int64_t N, int64_t B, Packing *pk, int *passes, int *bpp) {
    int nb = 1, ib = 1;
    const int kb = key_bits(N, B);
    while (nb < 31 && (int64_t(1) << nb) < N) ++nb;
    while (ib < 62 && (int64_t(1) << ib) < E) ++ib;
    pk->kb = kb;
    pk->nb = nb;
    pk->ib = ib;
    pk->sk = sort_key(N, B);
    *passes = (kb + kMaxDigitBitsP - 1) / kMaxDigitBitsP;
    *bpp = (kb + *passes - 1) / *passes;
    return kb + nb + ib <= 64;
}

struct CsrWs {
    Payload buf[2];
    uint64_t *pbuf[2];  // packed elements
    float *pw[2];       // packed path: weights
    uint32_t *sorted_key;
    uint8_t *next_dig;  // packed path: the next pass's digit of every element
    uint32_t *hist;
    uint32_t *hist_scan;
    uint32_t *dstart;   // packed path: start of every digit of the last pass, and E
    size_t bytes;
};

CsrWs carve_csr(void *base, int64_t E, int64_t N, int64_t B, bool weighted) {
    int nb, passes, bpp;
    digit_plan(key_bits(N, B), &nb, &passes, &bpp);
    Packing pk;
    int ppasses, pbpp;
    const bool packed = packed_plan(E, N, B, &pk, &ppasses, &pbpp);
    if (packed) {
        passes = ppasses;
        bpp = pbpp;
    }
    const int64_t ntiles = (E + kTile - 1) / kTile;
    const int64_t nhist = ntiles << bpp;
    Carver c(base);
    CsrWs w{};
    for (int b = 0; b < 2; ++b) {
        const int64_t n = (passes >= 2 + b) ? E : 0;  // buffer 0 from two passes on, buffer 1 from three
        if (packed) {
            w.pbuf[b] = c.take<uint64_t>(n);
            w.pw[b] = weighted && n ? c.take<float>(n) : nullptr;
            continue;
        }
        w.buf[b].key = c.take<uint32_t>(n);
        w.buf[b].id = c.take<uint32_t>(n);
        w.buf[b].src = c.take<uint32_t>(n);
        w.buf[b].w = weighted && n ? c.take<float>(n) : nullptr;
    }
    w.sorted_key = c.take<uint32_t>(E);
    w.next_dig = c.take<uint8_t>(packed && passes >= 2 ? E : 0);
    w.hist = c.take<uint32_t>(nhist);
    w.hist_scan = c.take<uint32_t>(scan_workspace_elems(nhist));
    w.dstart = c.take<uint32_t>(packed ? kMaxRadixP + 1 : 0);
    w.bytes = c.used + 256;
    return w;
}

// ------------------------------------------------------ inverse permutation
// inv[perm[p]] = p for a permutation perm of [0, E) (the edge id of every CSR
// slot), with coalesced writes. The pairs (id, slot), packed as
// id << ib | slot, are partitioned stably by the id's bits above kInvLow with
// the packed radix passes above; block b of 2^kInvLow consecutive ids then
// holds exactly the pairs at [b 2^kInvLow, (b+1) 2^kInvLow), since every id
// occurs once. One workgroup per block scatters its pairs into LDS by the
// low id bits and writes that block of inv in order. (One 4-byte scatter per
// edge instead writes every entry as a 32-byte partial line past L2: 3.7 GB
// for the 115M edges of the large power-law graph.) A malformed permutation
// leaves some entries of its blocks unset; every access stays in bounds.
constexpr int kInvLow = 14;  // ids per block: 2^14 int32 slots, 64 KB of LDS
constexpr int kInvThreads = 1024;

__global__ __launch_bounds__(kInvThreads) void k_inverse_block(const uint64_t *__restrict__ words,
                                                               const int64_t *__restrict__ perm, int64_t E, int ib,
                                                               int32_t *__restrict__ inv) {
    __shared__ int32_t slot[1 << kInvLow];
    constexpr uint64_t kLowMask = (1u << kInvLow) - 1;
    const int64_t b0 = (int64_t)blockIdx.x << kInvLow;
    const int64_t n = (E - b0) < (1 << kInvLow) ? (E - b0) : (1 << kInvLow);
    const uint64_t idmask = (1ull << ib) - 1;
    for (int64_t k = threadIdx.x; k < n; k += kInvThreads) {
        uint64_t e, p;
        if (words) {
            const uint64_t w = words[b0 + k];
            e = w >> ib;
            p = w & idmask;
        } else {  // a single block: the pairs straight from perm
            e = static_cast<uint64_t>(perm[b0 + k]);
            p = static_cast<uint64_t>(b0 + k);
        }
        slot[e & kLowMask] = static_cast<int32_t>(p);
    }
    __syncthreads();
    for (int64_t k = threadIdx.x; k < n; k += kInvThreads) inv[b0 + k] = slot[k];
}

struct InvPlan {
    Packing pk;   // key: the whole id (ib bits), no node id, slot: ib bits
    int passes;   // radix passes over the id bits above kInvLow
    int maxbits;  // widest digit
    int64_t ntiles;
};

InvPlan inv_plan(int64_t E) {
    InvPlan q{};
    int ib = 1;
    while (ib < 31 && (int64_t(1) << ib) < E) ++ib;
    q.pk.kb = ib;
    q.pk.nb = 0;
    q.pk.ib = ib;
    q.pk.sk.bsize = 0;
    q.pk.sk.N = 0;
    q.pk.sk.tb = 31;
    const int hb = ib > kInvLow ? ib - kInvLow : 0;
    q.passes = (hb + kMaxDigitBitsP - 1) / kMaxDigitBitsP;
    q.maxbits = q.passes ? (hb + q.passes - 1) / q.passes : 0;
    q.ntiles = (E + kTile - 1) / kTile;
    return q;
}

struct InvWs {
    uint64_t *buf[2];
    uint8_t *next_dig;
    uint32_t *hist;
    uint32_t *hist_scan;
    size_t bytes;
};

InvWs carve_inv(void *base, int64_t E) {
    const InvPlan q = inv_plan(E);
    const int64_t nhist = q.passes ? (q.ntiles << q.maxbits) : 0;
    Carver c(base);
    InvWs w{};
    w.buf[0] = c.take<uint64_t>(q.passes >= 1 ? E : 0);
    w.buf[1] = c.take<uint64_t>(q.passes >= 2 ? E : 0);
    w.next_dig = c.take<uint8_t>(q.passes >= 2 ? E : 0);
    w.hist = c.take<uint32_t>(nhist);
    w.hist_scan = c.take<uint32_t>(nhist ? scan_workspace_elems(nhist) : 0);
    w.bytes = c.used + 256;
    return w;
}

}  // namespace

size_t inverse_perm_sorted_workspace(int64_t E) { return carve_inv(nullptr, E).bytes; }

int inverse_perm_sorted(const int64_t *perm, int64_t E, int32_t *inv, void *ws, size_t ws_bytes, hipStream_t s) {
    if (E == 0) return PYG_OK;
    if (E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    const InvWs w = carve_inv(ws, E);
    if (ws_bytes < w.bytes || !ws) return PYG_ERR_WORKSPACE;
    const InvPlan q = inv_plan(E);
    const uint64_t *pin = nullptr;
    int shift = kInvLow;
    for (int p = 0; p < q.passes; ++p) {
        const int bits = pass_bits(q.pk.kb - kInvLow, q.passes, p);
        const bool more = p + 1 < q.passes;
        const int nbits = more ? pass_bits(q.pk.kb - kInvLow, q.passes, p + 1) : 0;
        if (p == 0)
            k_radix_hist64<kHistTiles0, 1><<<(unsigned)((q.ntiles + kHistTiles0 - 1) / kHistTiles0), kSortBlock, 0, s>>>(
                perm, nullptr, nullptr, nullptr, E, shift, bits, q.ntiles, q.pk, w.hist);
        else
            k_radix_hist64<kHistTiles, kHistCopies><<<(unsigned)((q.ntiles + kHistTiles - 1) / kHistTiles), kSortBlock, 0,
                                                      s>>>(nullptr, nullptr, pin, w.next_dig, E, shift, bits, q.ntiles,
                                                           q.pk, w.hist);
        PYG_LAUNCH_CHECK();
        PYG_TRY(scan_u32(w.hist, w.hist, q.ntiles << bits, false, w.hist_scan, s));
        uint64_t *pout = w.buf[p & 1];
        k_radix_scatter64<<<(unsigned)q.ntiles, kSortBlock, 0, s>>>(p == 0 ? perm : nullptr, nullptr, nullptr, pin,
                                                                  nullptr, pout, nullptr, nullptr, nullptr, nullptr,
                                                                  nullptr, E, shift, bits, q.ntiles, w.hist, 0, q.pk,
                                                                  more ? w.next_dig : nullptr, shift + bits, nbits);
        PYG_LAUNCH_CHECK();
        pin = pout;
        shift += bits;
    }
    const int64_t nblocks = (E + (int64_t(1) << kInvLow) - 1) >> kInvLow;
    k_inverse_block<<<(unsigned)nblocks, kInvThreads, 0, s>>>(pin, perm, E, q.pk.ib, inv);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

size_t degree_workspace(int64_t E, int64_t N) { return hist_workspace(E, N); }

int count_targets_i64(const int64_t *dst, int64_t E, int64_t N, int64_t *out, void *ws, hipStream_t s) {
    return count_targets<int64_t>(dst, E, N, out, ws, s);
}

int count_targets_f64(const int64_t *dst, int64_t E, int64_t N, double *out, void *ws, hipStream_t s) {
    return count_targets<double>(dst, E, N, out, ws, s);
}

}  // namespace pyg

using namespace pyg;

extern "C" int pyg_degree_workspace(int64_t E, int64_t N, size_t *bytes) {
    if (E < 0 || N < 0 || !bytes) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = degree_workspace(E, N);
    return PYG_OK;
}

extern "C" int pyg_degree(const int64_t *edge_index, int64_t E, int64_t N, int64_t *deg, void *ws, size_t ws_bytes,
                          void *stream) {
    if (E < 0 || N < 0 || (E > 0 && !edge_index) || (N > 0 && !deg)) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (E > 0 && N == 0) return PYG_ERR_INVALID_ARG;
    if (ws_bytes < degree_workspace(E, N) || !ws) return PYG_ERR_WORKSPACE;
    return count_targets<int64_t>(edge_index + E, E, N, deg, ws, static_cast<hipStream_t>(stream));
}

namespace pyg {
namespace {
__global__ void k_rowptr_degree(const int64_t *__restrict__ rowptr, int64_t N, int64_t *__restrict__ deg) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x)
        deg[i] = rowptr[i + 1] - rowptr[i];
}
}  // namespace
}  // namespace pyg

extern "C" int pyg_degree_csr(const pyg_csr *csr, int64_t *deg, void *stream) {
    if (!csr || csr->N < 0 || !csr->rowptr || (csr->N > 0 && !deg)) return PYG_ERR_INVALID_ARG;
    if (csr->N == 0) return PYG_OK;
    k_rowptr_degree<<<grid_for(csr->N, kBlock * 4), kBlock, 0, static_cast<hipStream_t>(stream)>>>(csr->rowptr, csr->N,
                                                                                                    deg);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

extern "C" int pyg_coo_to_csr_workspace(int64_t E, int64_t N, size_t *bytes) {
    if (E < 0 || N < 0 || !bytes) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve_csr(nullptr, E, N, 1, true).bytes;
    return PYG_OK;
}

namespace {

// The stable sort of the edges by sort key (target, or source block then
// target), carrying edge id, source and weight; rowptr over the B * N rows
// from the key changes of the sorted keys.
int coo_to_csr_impl(const int64_t *edge_index, int64_t E, int64_t N, int64_t B, const float *edge_weight,
                    int64_t *rowptr, int32_t *col, int64_t *perm, float *weight_csr, void *ws, size_t ws_bytes,
                    hipStream_t s) {
    if (!edge_weight) weight_csr = nullptr;
    const CsrWs w = carve_csr(ws, E, N, B, edge_weight != nullptr);
    if (ws_bytes < w.bytes || (w.bytes > 256 && !ws)) return PYG_ERR_WORKSPACE;
    const int64_t rows = B * N;
    if (E == 0) return fill<int64_t>(rowptr, rows + 1, 0, s);
    const int64_t *src = edge_index;
    const int64_t *dst = edge_index + E;

    const int64_t ntiles = (E + kTile - 1) / kTile;
    Packing pk;
    int ppasses, pbpp;
    if (packed_plan(E, N, B, &pk, &ppasses, &pbpp)) {
        const uint64_t *pin = nullptr;
        const float *pin_w = nullptr;
        int shift = 0;
        // the last pass's digit and the key bits below it (2-byte sorted keys if at most 16)
        const int last_bits = pass_bits(pk.kb, ppasses, ppasses - 1);
        const int low_bits = pk.kb - last_bits;
        const bool low_keys = low_bits <= 16;
        for (int p = 0; p < ppasses; ++p) {
            const int bits = pass_bits(pk.kb, ppasses, p);
            const bool last = p == ppasses - 1;
            const int64_t nhist = ntiles << bits;
            if (p == 0)
                k_radix_hist64<kHistTiles0, 1><<<(unsigned)((ntiles + kHistTiles0 - 1) / kHistTiles0), kSortBlock, 0, s>>>(
                    dst, src, pin, nullptr, E, shift, bits, ntiles, pk, w.hist);
            else
                k_radix_hist64<kHistTiles, kHistCopies><<<(unsigned)((ntiles + kHistTiles - 1) / kHistTiles), kSortBlock, 0,
                                                          s>>>(nullptr, src, pin, w.next_dig, E, shift, bits, ntiles, pk,
                                                               w.hist);
            PYG_LAUNCH_CHECK();
            PYG_TRY(scan_u32(w.hist, w.hist, nhist, false, w.hist_scan, s));
            uint64_t *pout = last ? nullptr : w.pbuf[p & 1];
            float *pout_w = last ? nullptr : w.pw[p & 1];
            const int nshift = shift + bits;
            const int nbits = last ? 0 : pass_bits(pk.kb, ppasses, p + 1);
            k_radix_scatter64<<<(unsigned)ntiles, kSortBlock, 0, s>>>(p == 0 ? dst : nullptr, src, edge_weight, pin, pin_w,
                                                                pout, pout_w, perm, col, weight_csr, w.sorted_key, E,
                                                                shift, bits, ntiles, w.hist, last ? (low_keys ? 2 : 1) : 0,
                                                                pk, last ? nullptr : w.next_dig, nshift, nbits);
            PYG_LAUNCH_CHECK();
            pin = pout;
            pin_w = pout_w;
            shift += bits;
        }
        if (low_keys) {
            k_digit_starts<<<1, kBlock, 0, s>>>(w.hist, ntiles, 1 << last_bits, E, w.dstart);
            PYG_LAUNCH_CHECK();
            k_row_bounds_low<<<grid_for(E + 1, kBlock * kRowBoundsLowSlots, int64_t(1) << 30), kBlock, 0, s>>>(
                reinterpret_cast<const uint16_t *>(w.sorted_key), w.dstart, 1 << last_bits, low_bits, pk.sk, E, rows,
                rowptr);
        } else {
            k_row_bounds<<<grid_for(E + 1, kBlock * 8, int64_t(1) << 30), kBlock, 0, s>>>(w.sorted_key, E, rows,
                                                                                         rowptr);
        }
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    int nb, passes, bpp;
    digit_plan(key_bits(N, B), &nb, &passes, &bpp);
    const SortKey sk = sort_key(N, B);
    Payload in{}, none{};
    int shift = 0;
    for (int p = 0; p < passes; ++p) {
        const int bits = (nb - shift) < bpp ? (nb - shift) : bpp;
        const bool last = p == passes - 1;
        const int64_t nhist = ntiles << bits;
        k_radix_hist<<<(unsigned)ntiles, kSortBlock, 0, s>>>(p == 0 ? dst : nullptr, src, in.key, sk, E, shift, bits,
                                                             ntiles, w.hist);
        PYG_LAUNCH_CHECK();
        PYG_TRY(scan_u32(w.hist, w.hist, nhist, false, w.hist_scan, s));
        Payload out = last ? none : w.buf[p & 1];
        if (last) out.key = w.sorted_key;
        k_radix_scatter<<<(unsigned)ntiles, kSortBlock, 0, s>>>(p == 0 ? dst : nullptr, src, edge_weight, in, out, perm,
                                                           col, weight_csr, E, shift, bits, ntiles, w.hist, last ? 1 : 0,
                                                           sk);
        PYG_LAUNCH_CHECK();
        in = out;
        shift += bits;
    }
    k_row_bounds<<<grid_for(E + 1, kBlock * 8, int64_t(1) << 30), kBlock, 0, s>>>(w.sorted_key, E, rows, rowptr);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

// deg[i] = the slots of target i over all source blocks.
__global__ void k_blocks_degree(const int64_t *__restrict__ rowptr, int64_t N, int64_t B, int64_t *__restrict__ deg) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t d = 0;
        for (int64_t b = 0; b < B; ++b) d += rowptr[b * N + i + 1] - rowptr[b * N + i];
        deg[i] = d;
    }
}

}  // namespace

extern "C" int pyg_coo_to_csr(const int64_t *edge_index, int64_t E, int64_t N, const float *edge_weight,
                              int64_t *rowptr, int32_t *col, int64_t *perm, float *weight_csr,
                              void *ws, size_t ws_bytes, void *stream) {
    if (E < 0 || N < 0 || !rowptr) return PYG_ERR_INVALID_ARG;
    if (E > 0 && (!edge_index || !col || !perm || N == 0)) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    return coo_to_csr_impl(edge_index, E, N, 1, edge_weight, rowptr, col, perm, weight_csr, ws, ws_bytes,
                           static_cast<hipStream_t>(stream));
}

extern "C" int pyg_coo_to_csr_blocked_workspace(int64_t E, int64_t N, int64_t B, size_t *bytes) {
    if (E < 0 || N < 0 || !bytes || B < 2 || B > 32) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31) || B * N >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve_csr(nullptr, E, N, B, true).bytes;
    return PYG_OK;
}

extern "C" int pyg_coo_to_csr_blocked(const int64_t *edge_index, int64_t E, int64_t N, int64_t B,
                                      const float *edge_weight, int64_t *rowptr, int32_t *col, int64_t *perm,
                                      float *weight_csr, void *ws, size_t ws_bytes, void *stream) {
    if (E < 0 || N < 0 || !rowptr || B < 2 || B > 32) return PYG_ERR_INVALID_ARG;
    if (E > 0 && (!edge_index || !col || N == 0)) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31) || B * N >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    return coo_to_csr_impl(edge_index, E, N, B, edge_weight, rowptr, col, perm, weight_csr, ws, ws_bytes,
                           static_cast<hipStream_t>(stream));
}

extern "C" int pyg_degree_csr_blocks(const pyg_csr_blocks *bcsr, int64_t *deg, void *stream) {
    if (!bcsr || !bcsr->rowptr || bcsr->N < 0 || bcsr->B < 2 || bcsr->B > 32 || (bcsr->N > 0 && !deg))
        return PYG_ERR_INVALID_ARG;
    if (bcsr->N == 0) return PYG_OK;
    k_blocks_degree<<<grid_for(bcsr->N, kBlock * 4), kBlock, 0, static_cast<hipStream_t>(stream)>>>(
        bcsr->rowptr, bcsr->N, bcsr->B, deg);
    PYG_LAUNCH_CHECK();
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

extern "C" int pyg_gather_edges(const int64_t *perm, int64_t E, const float *in, float *out, void *stream) {
    if (E < 0 || (E > 0 && (!perm || !in || !out))) return PYG_ERR_INVALID_ARG;
    if (E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (E > 0 && in == out) return PYG_ERR_INVALID_ARG;
    if (E == 0) return PYG_OK;
    k_gather_edges<<<grid_for(E, kBlock * 4), kBlock, 0, static_cast<hipStream_t>(stream)>>>(perm, E, in, out);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}
