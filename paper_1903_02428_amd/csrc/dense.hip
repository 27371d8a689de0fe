// Dense feature transform of a GCN layer, out = X Theta, on the matrix cores
// of gfx950 (v_mfma_f32_16x16x32_bf16: bf16 operands, fp32 accumulation;
// fp32 operands on v_mfma_f32_16x16x4_f32, below).
//
// Shapes on this path are tall and thin (N ~ 10^5 rows, Fi and Fo ~ 10^2),
// so the transform is bound by reading X and writing out, not by the matrix
// cores: every element of X is loaded exactly once, by one wavefront, in
// 16-byte pieces, and Theta (tens of KB) is staged in LDS per workgroup.
//
// Work split: a workgroup owns 128 rows (4 wavefronts x 32 rows) and 128
// output columns; each wavefront keeps 2 x 8 tiles of 16 x 16 fp32
// accumulators. Theta is first transposed and zero-padded to Theta^T
// [Fo_pad, Kp] (bf16, Kp a multiple of 32) so a lane's operand (8
// consecutive k of one column) is one 16-byte LDS read. K is processed in
// chunks of 128: the chunk's X operands of the wavefront are all loaded
// before the first multiply, so 8 x 16 bytes per lane are in flight.
//
// MFMA operand layout used (16 x 16 x 32): lane l supplies row l % 16 of A
// and column l % 16 of B with the 8 k values 8 (l / 16) .. 8 (l / 16) + 7;
// the 16 x 16 result gives lane l column l % 16, rows 4 (l / 16) .. +3.
// The product is formed transposed, out^T = Theta^T X^T (A = Theta^T from
// LDS, B = X^T, whose column is a row of X read as 16 contiguous bytes), so a
// lane ends with 4 consecutive output features of one node and stores them
// as one 16-byte (fp32) or 8-byte (bf16) write.
#include "common.hpp"

namespace pyg {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowsWave = 32;  // two 16-row tiles per wavefront
constexpr int kCols = 128;     // eight 16-column tiles per workgroup pass
constexpr int kChunk = 128;    // K per LDS stage
constexpr int kLdsStride = kChunk + 8;  // bf16 per LDS row; +16 B skews the banks
constexpr int64_t kPersistBlocks = 1024;  // 4 workgroups per CU

// Theta [Fi, Fo] -> Theta^T [Fo_pad, Kp], zero padded.
__global__ void k_theta_t(const uint16_t *__restrict__ theta, int64_t Fi, int64_t Fo, int64_t Kp, int64_t Fo_pad,
                          uint16_t *__restrict__ tt) {
    const int64_t n = Fo_pad * Kp;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t o = i / Kp, k = i % Kp;
        tt[i] = (o < Fo && k < Fi) ? theta[k * Fo + o] : uint16_t(0);
    }
}

union Frag {
    uint4 u;
    bf16x8 v;
};

// One 16-byte A operand: row `row`, k = k0 .. k0+7 (zeros outside the matrix).
// VEC: Fi % 8 == 0 and 16-byte aligned rows, so the 8 values are one load.
template <bool VEC>
__device__ __forceinline__ uint4 load_a(const uint16_t *__restrict__ x, int64_t N, int64_t Fi, int64_t row, int64_t k0) {
    if (row >= N || k0 >= Fi) return make_uint4(0, 0, 0, 0);
    const uint16_t *p = x + row * Fi + k0;
    if constexpr (VEC) {
        return *reinterpret_cast<const uint4 *>(p);
    } else {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t lo = (k0 + 2 * i < Fi) ? p[2 * i] : 0u;
            const uint32_t hi = (k0 + 2 * i + 1 < Fi) ? p[2 * i + 1] : 0u;
            w[i] = lo | (hi << 16);
        }
        return make_uint4(w[0], w[1], w[2], w[3]);
    }
}

// Store a wavefront's 32 x 128 tile: lane holds node r0 + 16t + li and
// output features c0 + 16u + 4lg + j (j = 0..3).
template <typename TO>
__device__ __forceinline__ void store_tile(TO *__restrict__ out, int64_t N, int64_t Fo, int64_t r0, int64_t c0, int li,
                                           int lg, const f32x4 (&acc)[2][8]) {
    const bool vec_out = (Fo & 3) == 0 && (reinterpret_cast<uintptr_t>(out) & (4 * sizeof(TO) - 1)) == 0;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int64_t row = r0 + 16 * t + li;
        if (row >= N) continue;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t col = c0 + 16 * u + 4 * lg;
            if (col >= Fo) continue;
            TO *o = out + row * Fo + col;
            if (vec_out && col + 4 <= Fo) {
                if constexpr (sizeof(TO) == 4) {
                    *reinterpret_cast<float4 *>(o) = make_float4(acc[t][u][0], acc[t][u][1], acc[t][u][2], acc[t][u][3]);
                } else {
                    const uint32_t lo = uint32_t(f32_to_bf16_rne(acc[t][u][0])) | (uint32_t(f32_to_bf16_rne(acc[t][u][1])) << 16);
                    const uint32_t hi = uint32_t(f32_to_bf16_rne(acc[t][u][2])) | (uint32_t(f32_to_bf16_rne(acc[t][u][3])) << 16);
                    *reinterpret_cast<uint2 *>(o) = make_uint2(lo, hi);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (col + j >= Fo) break;
                    if constexpr (sizeof(TO) == 4) o[j] = acc[t][u][j];
                    else o[j] = f32_to_bf16_rne(acc[t][u][j]);
                }
            }
        }
    }
}

// Stage Theta^T[c0 .. c0+127][kc .. kc+kn) in LDS (zeros past Fo), 16 B per thread and step.
__device__ __forceinline__ void stage_theta(uint16_t *lds, const uint16_t *__restrict__ tt, int64_t Fo, int64_t Kp,
                                            int64_t c0, int64_t kc, int kn) {
    const int per_row = kn / 8;
    for (int i = threadIdx.x; i < kCols * per_row; i += kBlock) {
        const int n = i / per_row, q = i % per_row;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (c0 + n < Fo) v = *reinterpret_cast<const uint4 *>(tt + (c0 + n) * Kp + kc + 8 * q);
        *reinterpret_cast<uint4 *>(lds + n * kLdsStride + 8 * q) = v;
    }
}

// Fi <= 128 (one K chunk): Theta^T is staged once and each workgroup walks
// over row blocks, loading the next block's X operands before multiplying
// the current ones.
template <typename TO, bool VEC>
__global__ __launch_bounds__(kBlock) void k_dense_small(const uint16_t *__restrict__ x, int64_t N, int64_t Fi,
                                                        int64_t Kp, const uint16_t *__restrict__ tt, int64_t Fo,
                                                        TO *__restrict__ out, int64_t nblocks) {
    __shared__ __align__(16) uint16_t lds[kCols * kLdsStride];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t c0 = (int64_t)blockIdx.y * kCols;
    const int li = lane & 15, lg = lane >> 4;
    const int kn = static_cast<int>(Kp);
    stage_theta(lds, tt, Fo, Kp, c0, 0, kn);
    __syncthreads();
    constexpr int S = kChunk / 32;
    uint4 a[2][S], an[2][S];
    auto load_block = [&](int64_t b, uint4 (&dst)[2][S]) {
        const int64_t r0 = b * (kRowsWave * (kBlock / kWave)) + wave * kRowsWave;
#pragma unroll
        for (int st = 0; st < S; ++st)
#pragma unroll
            for (int t = 0; t < 2; ++t)
                dst[t][st] = (st * 32 < kn) ? load_a<VEC>(x, N, Fi, r0 + 16 * t + li, 32 * st + 8 * lg)
                                            : make_uint4(0, 0, 0, 0);
    };
    int64_t b = blockIdx.x;
    if (b < nblocks) load_block(b, a);
    for (; b < nblocks; b += gridDim.x) {
        if (b + gridDim.x < nblocks) load_block(b + gridDim.x, an);
        f32x4 acc[2][8];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int u = 0; u < 8; ++u) acc[t][u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < S; ++st) {
            if (st * 32 >= kn) break;
            Frag fa0, fa1;
            fa0.u = a[0][st];
            fa1.u = a[1][st];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                Frag fb;
                fb.u = *reinterpret_cast<const uint4 *>(lds + (16 * u + li) * kLdsStride + 32 * st + 8 * lg);
                acc[0][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb.v, fa0.v, acc[0][u], 0, 0, 0);
                acc[1][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb.v, fa1.v, acc[1][u], 0, 0, 0);
            }
        }
        store_tile(out, N, Fo, b * (kRowsWave * (kBlock / kWave)) + wave * kRowsWave, c0, li, lg, acc);
#pragma unroll
        for (int st = 0; st < S; ++st)
#pragma unroll
            for (int t = 0; t < 2; ++t) a[t][st] = an[t][st];
    }
}

template <typename TO, bool VEC>
__global__ __launch_bounds__(kBlock) void k_dense(const uint16_t *__restrict__ x, int64_t N, int64_t Fi, int64_t Kp,
                                                  const uint16_t *__restrict__ tt, int64_t Fo, TO *__restrict__ out) {
    __shared__ __align__(16) uint16_t lds[kCols * kLdsStride];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t r0 = (int64_t)blockIdx.x * (kRowsWave * (kBlock / kWave)) + wave * kRowsWave;
    const int64_t c0 = (int64_t)blockIdx.y * kCols;
    const int li = lane & 15, lg = lane >> 4;

    f32x4 acc[2][8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[t][u] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int64_t kc = 0; kc < Kp; kc += kChunk) {
        const int kn = static_cast<int>((Kp - kc) < kChunk ? (Kp - kc) : kChunk);  // multiple of 32
        // this chunk's X operands first: 2 row tiles x kn/32 steps, 16 B each
        uint4 a[2][kChunk / 32];
#pragma unroll
        for (int s = 0; s < kChunk / 32; ++s)
#pragma unroll
            for (int t = 0; t < 2; ++t)
                a[t][s] = (s * 32 < kn) ? load_a<VEC>(x, N, Fi, r0 + 16 * t + li, kc + 32 * s + 8 * lg)
                                        : make_uint4(0, 0, 0, 0);
        __syncthreads();
        stage_theta(lds, tt, Fo, Kp, c0, kc, kn);
        __syncthreads();
#pragma unroll
        for (int s = 0; s < kChunk / 32; ++s) {
            if (s * 32 >= kn) break;
            Frag fa0, fa1;
            fa0.u = a[0][s];
            fa1.u = a[1][s];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                Frag fb;
                fb.u = *reinterpret_cast<const uint4 *>(lds + (16 * u + li) * kLdsStride + 32 * s + 8 * lg);
                acc[0][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb.v, fa0.v, acc[0][u], 0, 0, 0);
                acc[1][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb.v, fa1.v, acc[1][u], 0, 0, 0);
            }
        }
    }
    store_tile(out, N, Fo, r0, c0, li, lg, acc);
}

// ------------------------------------------------------------- fp32 operands
// The same tiling with fp32 X and Theta on v_mfma_f32_16x16x4_f32 (16 x 16 x
// 4, one k per lane group). A lane loads 16 bytes (4 consecutive k) of its X
// row and of its Theta^T row and feeds them to four MFMA steps: at step e,
// lane group lg holds k = 16 s + 4 lg + e in both operands, so the four
// steps cover the 16 k of the block with A and B paired on the same k (the
// order of the k inside a block is a relabelling of the sum, which the
// matrix unit adds in fp32 either way). K is staged 64 at a time.
constexpr int kChunkF = 64;
#ifndef PYG_DENSE_F32_PERSIST
#define PYG_DENSE_F32_PERSIST 1
#endif
constexpr int kLdsStrideF = kChunkF + 4;  // floats per LDS row; +16 B skews the banks

__global__ void k_theta_t_f32(const float *__restrict__ theta, int64_t Fi, int64_t Fo, int64_t Kp, int64_t Fo_pad,
                              float *__restrict__ tt) {
    const int64_t n = Fo_pad * Kp;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t o = i / Kp, k = i % Kp;
        tt[i] = (o < Fo && k < Fi) ? theta[k * Fo + o] : 0.f;
    }
}

// X[row, k0 .. k0+3] (zeros outside the matrix); VEC: Fi % 4 == 0 and
// 16-byte aligned rows, so the 4 values are one load.
template <bool VEC>
__device__ __forceinline__ f32x4 load_af(const float *__restrict__ x, int64_t N, int64_t Fi, int64_t row, int64_t k0) {
    if (row >= N || k0 >= Fi) return f32x4{0.f, 0.f, 0.f, 0.f};
    const float *p = x + row * Fi + k0;
    if constexpr (VEC) {
        return *reinterpret_cast<const f32x4 *>(p);
    } else {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = (k0 + i < Fi) ? p[i] : 0.f;
        return v;
    }
}

template <typename TO, bool VEC>
__global__ __launch_bounds__(kBlock) void k_dense_f32(const float *__restrict__ x, int64_t N, int64_t Fi, int64_t Kp,
                                                      const float *__restrict__ tt, int64_t Fo, TO *__restrict__ out) {
    __shared__ __align__(16) float lds[kCols * kLdsStrideF];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t r0 = (int64_t)blockIdx.x * (kRowsWave * (kBlock / kWave)) + wave * kRowsWave;
    const int64_t c0 = (int64_t)blockIdx.y * kCols;
    const int li = lane & 15, lg = lane >> 4;

    f32x4 acc[2][8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[t][u] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int64_t kc = 0; kc < Kp; kc += kChunkF) {
        const int kn = static_cast<int>((Kp - kc) < kChunkF ? (Kp - kc) : kChunkF);  // multiple of 16
        f32x4 a[2][kChunkF / 16];
#pragma unroll
        for (int st = 0; st < kChunkF / 16; ++st)
#pragma unroll
            for (int t = 0; t < 2; ++t)
                a[t][st] = (st * 16 < kn) ? load_af<VEC>(x, N, Fi, r0 + 16 * t + li, kc + 16 * st + 4 * lg)
                                          : f32x4{0.f, 0.f, 0.f, 0.f};
        __syncthreads();
        // stage Theta^T[c0 .. c0+127][kc .. kc+kn) (zeros past Fo), 16 B per thread and step
        const int per_row = kn / 4;
        for (int i = threadIdx.x; i < kCols * per_row; i += kBlock) {
            const int n = i / per_row, q = i % per_row;
            f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
            if (c0 + n < Fo) v = *reinterpret_cast<const f32x4 *>(tt + (c0 + n) * Kp + kc + 4 * q);
            *reinterpret_cast<f32x4 *>(lds + n * kLdsStrideF + 4 * q) = v;
        }
        __syncthreads();
#pragma unroll
        for (int st = 0; st < kChunkF / 16; ++st) {
            if (st * 16 >= kn) break;
            // all eight Theta^T operands first, then the steps e outermost: the 16
            // accumulators are updated in turn, so no MFMA waits on the one before
            f32x4 b[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                b[u] = *reinterpret_cast<const f32x4 *>(lds + (16 * u + li) * kLdsStrideF + 16 * st + 4 * lg);
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    acc[0][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[u][e], a[0][st][e], acc[0][u], 0, 0, 0);
                    acc[1][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(b[u][e], a[1][st][e], acc[1][u], 0, 0, 0);
                }
        }
    }
    store_tile(out, N, Fo, r0, c0, li, lg, acc);
}

// Fi <= 128: persistent workgroups that stage the whole Theta^T (128 columns
// x Kp <= 128 fp32, 66 KB) once and walk over row blocks, loading the next
// block's X operands before multiplying the current ones, as the bf16 form.
constexpr int kLdsStrideFS = 128 + 4;
constexpr int64_t kPersistBlocksF = 512;  // 2 workgroups per CU (LDS)

template <typename TO, bool VEC>
__global__ __launch_bounds__(kBlock) void k_dense_small_f32(const float *__restrict__ x, int64_t N, int64_t Fi,
                                                            int64_t Kp, const float *__restrict__ tt, int64_t Fo,
                                                            TO *__restrict__ out, int64_t nblocks) {
    __shared__ __align__(16) float lds[kCols * kLdsStrideFS];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t c0 = (int64_t)blockIdx.y * kCols;
    const int li = lane & 15, lg = lane >> 4;
    const int kn = static_cast<int>(Kp);  // multiple of 16, at most 128
    const int per_row = kn / 4;
    for (int i = threadIdx.x; i < kCols * per_row; i += kBlock) {
        const int n = i / per_row, q = i % per_row;
        f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
        if (c0 + n < Fo) v = *reinterpret_cast<const f32x4 *>(tt + (c0 + n) * Kp + 4 * q);
        *reinterpret_cast<f32x4 *>(lds + n * kLdsStrideFS + 4 * q) = v;
    }
    __syncthreads();
    constexpr int S = 128 / 16;
    f32x4 a[2][S], an[2][S];
    auto load_block = [&](int64_t b, f32x4 (&dst)[2][S]) {
        const int64_t r0 = b * (kRowsWave * (kBlock / kWave)) + wave * kRowsWave;
#pragma unroll
        for (int st = 0; st < S; ++st)
#pragma unroll
            for (int t = 0; t < 2; ++t)
                dst[t][st] = (st * 16 < kn) ? load_af<VEC>(x, N, Fi, r0 + 16 * t + li, 16 * st + 4 * lg)
                                            : f32x4{0.f, 0.f, 0.f, 0.f};
    };
    int64_t b = blockIdx.x;
    if (b < nblocks) load_block(b, a);
    for (; b < nblocks; b += gridDim.x) {
        if (b + gridDim.x < nblocks) load_block(b + gridDim.x, an);
        f32x4 acc[2][8];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int u = 0; u < 8; ++u) acc[t][u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < S; ++st) {
            if (st * 16 >= kn) break;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const f32x4 bv = *reinterpret_cast<const f32x4 *>(lds + (16 * u + li) * kLdsStrideFS + 16 * st + 4 * lg);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[0][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv[e], a[0][st][e], acc[0][u], 0, 0, 0);
                    acc[1][u] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv[e], a[1][st][e], acc[1][u], 0, 0, 0);
                }
            }
        }
        store_tile(out, N, Fo, b * (kRowsWave * (kBlock / kWave)) + wave * kRowsWave, c0, li, lg, acc);
#pragma unroll
        for (int st = 0; st < S; ++st)
#pragma unroll
            for (int t = 0; t < 2; ++t) a[t][st] = an[t][st];
    }
}

int64_t kpad(int64_t Fi) { return (Fi + 31) / 32 * 32; }
int64_t kpadf(int64_t Fi) { return (Fi + 15) / 16 * 16; }
int64_t fopad(int64_t Fo) { return (Fo + 15) / 16 * 16; }

}  // namespace
}  // namespace pyg

using namespace pyg;

extern "C" int pyg_dense_transform_workspace(int64_t Fi, int64_t Fo, size_t *bytes) {
    if (!bytes || Fi < 0 || Fo < 0) return PYG_ERR_INVALID_ARG;
    if (Fi >= (int64_t(1) << 24) || Fo >= (int64_t(1) << 24)) return PYG_ERR_UNSUPPORTED;
    // Theta^T padded: bf16 (K to 32) or fp32 (K to 16), whichever is larger
    const size_t b16 = static_cast<size_t>(fopad(Fo) * kpad(Fi)) * 2, b32 = static_cast<size_t>(fopad(Fo) * kpadf(Fi)) * 4;
    *bytes = align_up(b16 > b32 ? b16 : b32, 256);
    return PYG_OK;
}

extern "C" int pyg_dense_transform(const void *x, int x_dtype, int64_t N, int64_t Fi, const void *theta, int64_t Fo,
                                   void *out, int out_dtype, void *ws, size_t ws_bytes, void *stream) {
    if (N < 0 || Fi < 0 || Fo < 0) return PYG_ERR_INVALID_ARG;
    if (x_dtype != PYG_BF16 && x_dtype != PYG_F32) return PYG_ERR_INVALID_ARG;
    if (out_dtype != PYG_BF16 && out_dtype != PYG_F32) return PYG_ERR_INVALID_ARG;
    if (N >= (int64_t(1) << 31)) return PYG_ERR_UNSUPPORTED;
    if (N * Fo > 0 && !out) return PYG_ERR_INVALID_ARG;
    if (N * Fi > 0 && !x) return PYG_ERR_INVALID_ARG;
    if (Fi * Fo > 0 && !theta) return PYG_ERR_INVALID_ARG;
    size_t need;
    PYG_TRY(pyg_dense_transform_workspace(Fi, Fo, &need));
    if (N * Fo == 0) return PYG_OK;
    if (!ws || ws_bytes < need) return PYG_ERR_WORKSPACE;
    const int64_t osz = out_dtype == PYG_F32 ? 4 : 2, xsz = x_dtype == PYG_F32 ? 4 : 2;
    const char *xb = static_cast<const char *>(x);
    const char *ob = static_cast<const char *>(out);
    if (ob < xb + N * Fi * xsz && xb < ob + N * Fo * osz) return PYG_ERR_INVALID_ARG;  // out overlaps x
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (x_dtype == PYG_F32) {
        const int64_t Kp = kpadf(Fi), Fp = fopad(Fo);
        float *tt = static_cast<float *>(ws);
        k_theta_t_f32<<<grid_for(Fp * Kp, kBlock * 4), kBlock, 0, s>>>(static_cast<const float *>(theta), Fi, Fo, Kp, Fp,
                                                                       tt);
        PYG_LAUNCH_CHECK();
        const bool vec = Fi % 4 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
        const int64_t nblocks = (N + kRowsWave * (kBlock / kWave) - 1) / (kRowsWave * (kBlock / kWave));
        const unsigned gy = static_cast<unsigned>((Fo + kCols - 1) / kCols);
        const dim3 grid(static_cast<unsigned>(nblocks), gy);
        const float *xf = static_cast<const float *>(x);
        if (Kp <= 128 && PYG_DENSE_F32_PERSIST) {  // persistent workgroups, Theta staged once
            const int64_t iters = (nblocks + kPersistBlocksF - 1) / kPersistBlocksF;
            const dim3 g(static_cast<unsigned>((nblocks + iters - 1) / iters), gy);
            if (out_dtype == PYG_F32) {
                if (vec) k_dense_small_f32<float, true><<<g, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<float *>(out), nblocks);
                else k_dense_small_f32<float, false><<<g, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<float *>(out), nblocks);
            } else {
                if (vec) k_dense_small_f32<uint16_t, true><<<g, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out), nblocks);
                else k_dense_small_f32<uint16_t, false><<<g, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out), nblocks);
            }
            PYG_LAUNCH_CHECK();
            return PYG_OK;
        }
        if (out_dtype == PYG_F32) {
            if (vec) k_dense_f32<float, true><<<grid, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<float *>(out));
            else k_dense_f32<float, false><<<grid, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<float *>(out));
        } else {
            if (vec) k_dense_f32<uint16_t, true><<<grid, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out));
            else k_dense_f32<uint16_t, false><<<grid, kBlock, 0, s>>>(xf, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out));
        }
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    const int64_t Kp = kpad(Fi), Fp = fopad(Fo);
    uint16_t *tt = static_cast<uint16_t *>(ws);
    k_theta_t<<<grid_for(Fp * Kp, kBlock * 4), kBlock, 0, s>>>(static_cast<const uint16_t *>(theta), Fi, Fo, Kp, Fp, tt);
    PYG_LAUNCH_CHECK();
    const bool vec = Fi % 8 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
    const int64_t nblocks = (N + kRowsWave * (kBlock / kWave) - 1) / (kRowsWave * (kBlock / kWave));
    const unsigned gy = static_cast<unsigned>((Fo + kCols - 1) / kCols);
    const uint16_t *xx = static_cast<const uint16_t *>(x);
    if (Kp <= kChunk) {  // persistent workgroups, Theta staged once
        const int64_t iters = (nblocks + kPersistBlocks - 1) / kPersistBlocks;  // the same count for every workgroup
        const dim3 g(static_cast<unsigned>((nblocks + iters - 1) / iters), gy);
        if (out_dtype == PYG_F32) {
            if (vec) k_dense_small<float, true><<<g, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<float *>(out), nblocks);
            else k_dense_small<float, false><<<g, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<float *>(out), nblocks);
        } else {
            if (vec) k_dense_small<uint16_t, true><<<g, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out), nblocks);
            else k_dense_small<uint16_t, false><<<g, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out), nblocks);
        }
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    const dim3 grid(static_cast<unsigned>(nblocks), gy);
    if (out_dtype == PYG_F32) {
        if (vec) k_dense<float, true><<<grid, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<float *>(out));
        else k_dense<float, false><<<grid, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<float *>(out));
    } else {
        if (vec) k_dense<uint16_t, true><<<grid, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out));
        else k_dense<uint16_t, false><<<grid, kBlock, 0, s>>>(xx, N, Fi, Kp, tt, Fo, static_cast<uint16_t *>(out));
    }
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}
