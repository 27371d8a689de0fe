// Device-wide prefix sum (reduce-then-scan, no inter-workgroup waiting).
// Used for CSR row pointers and radix-sort digit offsets.
#include "common.hpp"

namespace pyg {
namespace {

constexpr int kItems = 8;                     // consecutive elements per thread
constexpr int64_t kSeg = kBlock * kItems;     // elements per workgroup

template <typename T>
__device__ __forceinline__ T wave_inclusive_scan(T v, int lane) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        T y = __shfl_up(v, d, kWave);
        if (lane >= d) v += y;
    }
    return v;
}

// Exclusive scan of one value per thread across the workgroup; returns the
// thread's exclusive prefix and writes the workgroup total.
template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T *lds, T *total) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    T incl = wave_inclusive_scan(v, lane);
    if (lane == kWave - 1) lds[wave] = incl;
    __syncthreads();
    T before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kBlock / kWave; ++w) {
        T t = lds[w];
        if (w < wave) before += t;
        all += t;
    }
    __syncthreads();
    *total = all;
    return before + incl - v;
}

// A thread's kItems consecutive elements, as 16-byte loads when they are
// all in range and the array is 16-byte aligned (each thread's run starts at
// a multiple of kItems elements).
template <typename T>
__device__ __forceinline__ void load_items(const T *p, int64_t base, int64_t n, T (&v)[kItems]) {
    static_assert((kItems * sizeof(T)) % 16 == 0, "whole 16-byte loads per thread");
    if (base + kItems <= n && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
#pragma unroll
        for (int i = 0; i < kItems; i += 16 / (int)sizeof(T)) {
            const uint4 q = *reinterpret_cast<const uint4 *>(p + base + i);
            __builtin_memcpy(&v[i], &q, 16);
        }
    } else {
#pragma unroll
        for (int i = 0; i < kItems; ++i) v[i] = (base + i < n) ? p[base + i] : T(0);
    }
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_reduce(const T *__restrict__ in, int64_t n, T *__restrict__ sums) {
    __shared__ T lds[kBlock / kWave];
    const int64_t base = blockIdx.x * kSeg + (int64_t)threadIdx.x * kItems;
    T v[kItems];
    load_items(in, base, n, v);
    T s = 0;
#pragma unroll
    for (int i = 0; i < kItems; ++i) s += v[i];
    T total;
    block_exclusive_scan(s, lds, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_apply(const T *in, T *out, int64_t n,
                                                       const T *__restrict__ offsets, bool inclusive) {
    __shared__ T lds[kBlock / kWave];
    const int64_t base = blockIdx.x * kSeg + (int64_t)threadIdx.x * kItems;
    T v[kItems];
    load_items(in, base, n, v);
    T s = 0;
#pragma unroll
    for (int i = 0; i < kItems; ++i) s += v[i];
    T total;
    T run = block_exclusive_scan(s, lds, &total) + (offsets ? offsets[blockIdx.x] : T(0));
    T r[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const T next = run + v[i];
        r[i] = inclusive ? next : run;
        run = next;
    }
    if (base + kItems <= n && (reinterpret_cast<uintptr_t>(out) & 15) == 0) {
#pragma unroll
        for (int i = 0; i < kItems; i += 16 / (int)sizeof(T)) {
            uint4 q;
            __builtin_memcpy(&q, &r[i], 16);
            *reinterpret_cast<uint4 *>(out + base + i) = q;
        }
    } else {
#pragma unroll
        for (int i = 0; i < kItems; ++i)
            if (base + i < n) out[base + i] = r[i];
    }
}

template <typename T>
int scan_impl(const T *in, T *out, int64_t n, bool inclusive, T *ws, hipStream_t s) {
    if (n <= 0) return PYG_OK;
    const int64_t blocks = (n + kSeg - 1) / kSeg;
    if (blocks == 1) {
        k_scan_apply<T><<<1, kBlock, 0, s>>>(in, out, n, nullptr, inclusive);
        PYG_LAUNCH_CHECK();
        return PYG_OK;
    }
    T *sums = ws;
    T *rest = ws + align_up(blocks, 64);
    k_scan_reduce<T><<<(unsigned)blocks, kBlock, 0, s>>>(in, n, sums);
    PYG_LAUNCH_CHECK();
    PYG_TRY(scan_impl<T>(sums, sums, blocks, false, rest, s));
    k_scan_apply<T><<<(unsigned)blocks, kBlock, 0, s>>>(in, out, n, sums, inclusive);
    PYG_LAUNCH_CHECK();
    return PYG_OK;
}

}  // namespace

size_t scan_workspace_elems(int64_t n) {
    const int64_t blocks = (n + kSeg - 1) / kSeg;
    if (blocks <= 1) return 0;
    return align_up(blocks, 64) + scan_workspace_elems(blocks);
}

int scan_u32(const uint32_t *in, uint32_t *out, int64_t n, bool inclusive, uint32_t *ws, hipStream_t s) {
    return scan_impl<uint32_t>(in, out, n, inclusive, ws, s);
}

int scan_i64(const int64_t *in, int64_t *out, int64_t n, bool inclusive, int64_t *ws, hipStream_t s) {
    return scan_impl<int64_t>(in, out, n, inclusive, ws, s);
}

}  // namespace pyg
