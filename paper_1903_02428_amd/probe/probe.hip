// Bandwidth probes for the roofline of the propagate kernels on gfx950
// (measurement infrastructure, not part of the propagate library's ABI).
//
//   pyg_probe_flush        writes `bytes` of a buffer (>= 1 GiB evicts every
//                          XCD's L2 and the 256 MB Infinity Cache);
//   pyg_probe_gather       reads n random cache lines (64 or 128 bytes) of a
//                          buffer: exactly n * line_bytes bytes are requested,
//                          with no index stream (line numbers come from a
//                          hash of the gather's counter). With parts = 8 the
//                          workgroups of XCD x (workgroup w runs on XCD w % 8)
//                          draw only from the x-th eighth of the buffer, the
//                          pattern of an XCD-affine gather (groups should
//                          then be a multiple of 8);
//   pyg_probe_stream_read  reads a buffer once, front to back;
//   pyg_probe_atomic       n random 256-byte blocks of a float buffer each
//                          get a float atomic add per element (no return).
//
// Every kernel writes one 4-byte word per thread into `sink` (the xor of what
// it loaded), so no load can be dropped; the sink holds
// pyg_probe_sink_elems() words. All calls are asynchronous on `stream` and
// return 0, or -1 for a bad argument, -4 for a failed launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;
constexpr int kGroups = 256 * 8;     // workgroups per launch (default): 8 per compute unit
constexpr int kMaxGroups = 256 * 32; // the sink holds one word per thread of this many
constexpr int kInFlight = 8;         // loads in flight per lane (streaming read)

// Integer hash of a 32-bit counter (the "lowbias32" mixer: xor-shift and
// multiply rounds); spreads consecutive counters over the whole range.
__device__ __forceinline__ uint32_t mix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

__global__ __launch_bounds__(kThreads) void k_flush(uint4 *__restrict__ buf, uint64_t n16, uint32_t salt) {
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    for (uint64_t i = blockIdx.x * (uint64_t)kThreads + threadIdx.x; i < n16; i += stride) {
        const uint32_t v = static_cast<uint32_t>(i) ^ salt;
        buf[i] = make_uint4(v, v + 1, v + 2, v + 3);
    }
}

// LANES lanes (16 bytes each) read one line of LANES * 16 bytes per gather;
// every lane keeps U gathers in flight.
template <int LANES, int U>
__global__ __launch_bounds__(kThreads) void k_gather(const uint4 *__restrict__ buf, uint32_t draws_per_part,
                                                     uint64_t lines_per_part, int parts, uint32_t stride,
                                                     uint64_t n_gathers, uint32_t seed, uint32_t *__restrict__ sink) {
    const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
    const uint32_t sub = threadIdx.x & (LANES - 1);
    const uint64_t group = tid / LANES;
    const uint64_t ngroups = (uint64_t)gridDim.x * (kThreads / LANES);
    const uint64_t base = (uint64_t)(parts > 1 ? blockIdx.x % parts : 0) * lines_per_part;
    uint32_t acc = 0;
    for (uint64_t k0 = group; k0 < n_gathers; k0 += ngroups * U) {
        uint4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t k = k0 + (uint64_t)u * ngroups;
            v[u] = make_uint4(0, 0, 0, 0);
            if (k < n_gathers) {
                const uint64_t line =
                    base + stride * (((uint64_t)mix32(static_cast<uint32_t>(k) ^ seed) * draws_per_part) >> 32);
                v[u] = buf[line * LANES + sub];
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    sink[tid] = acc;
}

__global__ __launch_bounds__(kThreads) void k_stream(const uint4 *__restrict__ buf, uint64_t n16,
                                                     uint32_t *__restrict__ sink) {
    const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    uint32_t acc = 0;
    for (uint64_t i0 = tid; i0 < n16; i0 += stride * kInFlight) {
        uint4 v[kInFlight];
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) {
            const uint64_t i = i0 + (uint64_t)u * stride;
            v[u] = i < n16 ? buf[i] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    sink[tid] = acc;
}

// Float atomic adds with no return: wavefront op k adds 1 to the 64
// consecutive floats (256 bytes, four 64-byte atomic requests) of a random
// 256-byte block of the buffer; ops are independent, so many are in flight.
// Exactly n_ops * 64 float adds.
__global__ __launch_bounds__(kThreads) void k_atomic(float *__restrict__ buf, uint32_t blocks, uint64_t n_ops,
                                                     uint32_t seed) {
    const int lane = threadIdx.x & 63;
    const uint64_t wave = (blockIdx.x * (uint64_t)kThreads + threadIdx.x) / 64;
    const uint64_t nw = (uint64_t)gridDim.x * (kThreads / 64);
    for (uint64_t k = wave; k < n_ops; k += nw) {
        const uint64_t b = ((uint64_t)mix32(static_cast<uint32_t>(k) ^ seed) * blocks) >> 32;
        unsafeAtomicAdd(buf + b * 64 + lane, 1.0f);
    }
}

int launched() { return hipGetLastError() == hipSuccess ? 0 : -4; }

}  // namespace

extern "C" int64_t pyg_probe_sink_elems(void) { return (int64_t)kMaxGroups * kThreads; }

extern "C" int pyg_probe_flush(void *buf, uint64_t bytes, uint32_t salt, void *stream) {
    if (!buf || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0) return -1;
    if (bytes == 0) return 0;
    k_flush<<<kGroups, kThreads, 0, static_cast<hipStream_t>(stream)>>>(static_cast<uint4 *>(buf), bytes / 16, salt);
    return launched();
}

// in_flight: gathers in flight per lane (4, 8 or 16); groups: workgroups of
// 256 threads (1 .. 8192); stride >= 1: only every stride-th line of a part
// is read (the lines of one feature window of wider rows).
extern "C" int pyg_probe_gather(const void *buf, uint64_t buf_bytes, int line_bytes, int parts, int stride,
                                uint64_t n_gathers, uint32_t seed, int in_flight, int groups, uint32_t *sink,
                                void *stream) {
    if (!buf || !sink || (line_bytes != 64 && line_bytes != 128) || (parts != 1 && parts != 8)) return -1;
    if ((in_flight != 4 && in_flight != 8 && in_flight != 16) || groups < 1 || groups > kMaxGroups) return -1;
    if (reinterpret_cast<uintptr_t>(buf) % line_bytes != 0 || n_gathers >= (uint64_t(1) << 32)) return -1;
    const uint64_t lines = buf_bytes / line_bytes;
    if (stride < 1) return -1;
    const uint64_t per_part = lines / parts;  // parts * per_part <= lines: every line index stays in the buffer
    // lines base + stride * r with r < per_part / stride stay inside the part
    if (per_part / stride == 0 || per_part >= (uint64_t(1) << 32)) return -1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const uint4 *b = static_cast<const uint4 *>(buf);
    const uint32_t pp = static_cast<uint32_t>(per_part / stride);
    const uint32_t st = static_cast<uint32_t>(stride);
    const uint64_t per = per_part;  // the part's first line is part * per_part
#define PYG_PROBE_GATHER(L, U) k_gather<L, U><<<groups, kThreads, 0, s>>>(b, pp, per, parts, st, n_gathers, seed, sink)
    if (line_bytes == 128) {
        if (in_flight == 4) PYG_PROBE_GATHER(8, 4);
        else if (in_flight == 8) PYG_PROBE_GATHER(8, 8);
        else PYG_PROBE_GATHER(8, 16);
    } else {
        if (in_flight == 4) PYG_PROBE_GATHER(4, 4);
        else if (in_flight == 8) PYG_PROBE_GATHER(4, 8);
        else PYG_PROBE_GATHER(4, 16);
    }
#undef PYG_PROBE_GATHER
    return launched();
}

extern "C" int pyg_probe_stream_read(const void *buf, uint64_t bytes, uint32_t *sink, void *stream) {
    if (!buf || !sink || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0) return -1;
    k_stream<<<kGroups, kThreads, 0, static_cast<hipStream_t>(stream)>>>(static_cast<const uint4 *>(buf), bytes / 16,
                                                                        sink);
    return launched();
}

extern "C" int pyg_probe_atomic(float *buf, uint64_t buf_bytes, uint64_t n_ops, uint32_t seed, void *stream) {
    if (!buf || reinterpret_cast<uintptr_t>(buf) % 256 != 0 || n_ops >= (uint64_t(1) << 32)) return -1;
    const uint64_t blocks = buf_bytes / 256;  // block b covers floats [64 b, 64 b + 64): inside the buffer
    if (blocks == 0 || blocks >= (uint64_t(1) << 32)) return -1;
    k_atomic<<<kGroups, kThreads, 0, static_cast<hipStream_t>(stream)>>>(buf, static_cast<uint32_t>(blocks), n_ops,
                                                                        seed);
    return launched();
}
