// Source-blocked CSR: the slots of every CSR row regrouped by the block of
// their source node (B blocks of ceil(N / B) consecutive node ids), keeping
// their order inside a block (ascending edge id). Virtual row b * N + i holds
// the slots of target i whose source lies in block b; rowptr is the exclusive
// prefix sum of the virtual rows' lengths in that order, so the result is
// itself a CSR over B * N rows. It is preprocessing of the propagate's
// XCD-affine form (one source block per L2), built once per graph.
//
// Three steps: count every row's slots per block (one wavefront per row,
// a ballot per block and batch of 64 slots), exclusive scan of the B * N
// counts, then every row writes its slots to their blocks' ranges (the
// same ballots give each slot its rank among the row's slots of its block).
#include "common.hpp"

namespace pyg {
namespace {

constexpr int kRowsPerBlock = kBlock / kWave;  // one wavefront per row

__device__ __forceinline__ int source_block(int32_t c, int64_t bsize) {
    return static_cast<int>(static_cast<uint32_t>(c) / static_cast<uint32_t>(bsize));
}

// cnt[b * N + i] = slots of row i with source block b.
__global__ __launch_bounds__(kBlock) void k_block_count(const int64_t *__restrict__ rowptr,
                                                         const int32_t *__restrict__ col, int64_t N, int B,
                                                         int64_t bsize, int64_t *__restrict__ cnt) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t nw = (int64_t)gridDim.x * kRowsPerBlock;
    for (int64_t i = blockIdx.x * (int64_t)kRowsPerBlock + threadIdx.x / kWave; i < N; i += nw) {
        const int64_t s = uniform64(rowptr[i]), t = uniform64(rowptr[i + 1]);
        int64_t mine = 0;  // lane b counts block b
        for (int64_t base = s; base < t; base += kWave) {
            const bool in = base + lane < t;
            const int blk = in ? source_block(col[base + lane], bsize) : -1;
            for (int b = 0; b < B; ++b) {
                const uint64_t m = __ballot(blk == b);
                if (lane == b) mine += __popcll(m);
            }
        }
        if (lane < B) cnt[(int64_t)lane * N + i] = mine;
    }
}

// Every row's slots to their blocks' ranges, in order inside each block.
__global__ __launch_bounds__(kBlock) void k_block_scatter(const int64_t *__restrict__ rowptr,
                                                           const int32_t *__restrict__ col,
                                                           const float *__restrict__ weight,
                                                           const int64_t *__restrict__ perm, int64_t N, int B,
                                                           int64_t bsize, const int64_t *__restrict__ brow,
                                                           int32_t *__restrict__ bcol, float *__restrict__ bweight,
                                                           int64_t *__restrict__ bperm) {
    const int lane = threadIdx.x & (kWave - 1);
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));  // lanes < this one
    const int64_t nw = (int64_t)gridDim.x * kRowsPerBlock;
    for (int64_t i = blockIdx.x * (int64_t)kRowsPerBlock + threadIdx.x / kWave; i < N; i += nw) {
        const int64_t s = uniform64(rowptr[i]), t = uniform64(rowptr[i + 1]);
        int64_t next = lane < B ? brow[(int64_t)lane * N + i] : 0;  // lane b: next free slot of block b
        for (int64_t base = s; base < t; base += kWave) {
            const bool in = base + lane < t;
            const int32_t c = in ? col[base + lane] : 0;
            const int blk = in ? source_block(c, bsize) : -1;
            int64_t dst = -1;
            for (int b = 0; b < B; ++b) {
                const uint64_t m = __ballot(blk == b);
                if (m == 0) continue;  // uniform
                const int64_t start = __shfl(next, b, kWave);
                if (blk == b) dst = start + __popcll(m & below);
                if (lane == b) next += __popcll(m);
            }
            if (in && dst >= 0) {  // dst < 0 only for a source id outside [0, N) (undefined input)
                bcol[dst] = c;
                if (bweight) bweight[dst] = weight[base + lane];
                if (bperm) bperm[dst] = perm[base + lane];
            }
        }
    }
}

struct BlocksWs {
    int64_t *scan;
    size_t bytes;
};

BlocksWs carve_blocks(void *base, int64_t N, int64_t B) {
    Carver c(base);
    BlocksWs w{};
    w.scan = c.take<int64_t>(scan_workspace_elems(B * N));
    w.bytes = c.used + 256;
    return w;
}

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" int pyg_csr_blocks_workspace(int64_t N, int64_t E, int64_t B, size_t *bytes) {
    if (!bytes || N < 0 || E < 0 || B < 2 || B > 32)
        return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    *bytes = carve_blocks(nullptr, N, B).bytes;
    return PYG_OK;
}

extern "C" int pyg_csr_blocks_build(const pyg_csr *csr, int64_t B, int64_t *rowptr, int32_t *col, int64_t *perm,
                                    float *weight, void *ws, size_t ws_bytes, void *stream) {
    if (!csr || !csr->rowptr || csr->N < 0 || csr->E < 0 || !rowptr) return PYG_ERR_INVALID_ARG;
    const int64_t N = csr->N, E = csr->E;
    size_t need = 0;
    PYG_TRY(pyg_csr_blocks_workspace(N, E, B, &need));
    if (E > 0 && (!csr->col || !col || N == 0)) return PYG_ERR_INVALID_ARG;
    if (perm && !csr->perm && E > 0) return PYG_ERR_INVALID_ARG;
    if (weight && !csr->weight && E > 0) return PYG_ERR_INVALID_ARG;
    if (ws_bytes < need || !ws) return PYG_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const BlocksWs w = carve_blocks(ws, N, B);
    const int64_t bsize = N > 0 ? (N + B - 1) / B : 1;
    const int64_t rows = B * N;
    if (rows > 0) {
        // counts into rowptr[0 .. B*N), then scanned in place
        k_block_count<<<grid_for(N, kRowsPerBlock, 1 << 16), kBlock, 0, s>>>(csr->rowptr, csr->col, N,
                                                                             static_cast<int>(B), bsize, rowptr);
        PYG_LAUNCH_CHECK();
        PYG_TRY(scan_i64(rowptr, rowptr, rows, false, w.scan, s));
    }
    PYG_TRY(fill<int64_t>(rowptr + rows, 1, E, s));
    if (E > 0) {
        k_block_scatter<<<grid_for(N, kRowsPerBlock, 1 << 16), kBlock, 0, s>>>(
            csr->rowptr, csr->col, weight ? csr->weight : nullptr, perm ? csr->perm : nullptr, N,
            static_cast<int>(B), bsize, rowptr, col, weight, perm);
        PYG_LAUNCH_CHECK();
    }
    return PYG_OK;
}
