// Allocation-free propagate: pyg_propagate with its scratch in a static
// device array instead of a caller workspace, for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid allocation).
//
// The array lives in this file's code object; every GPU the library runs on
// holds its own copy (kNoallocScratchBytes) until the process ends. Host code
// never passes the array's name to a kernel or a runtime call: in host code
// that name is only a stand-in for the symbol. Its device address is looked
// up once per device with hipGetSymbolAddress (that device current) and kept;
// the kernels receive that address as their workspace. The kernels clear
// what must start at zero themselves (fill kernels, no memset), so the
// contents left by an earlier call never matter. Calls that overlap in time
// on one GPU share the array and race.
#include <mutex>

#include "common.hpp"

namespace {

constexpr size_t kNoallocScratchBytes = size_t(PYG_NOALLOC_SCRATCH_MIB) << 20;  // from the public header
static_assert(kNoallocScratchBytes % 256 == 0, "scratch size");

__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device

// Device address of the current device's scratch array (resolved once).
int device_scratch(void *stream, void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return PYG_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return PYG_ERR_UNSUPPORTED;
    if (stream) {
        hipDevice_t sdev = -1;
        if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev) != hipSuccess) return PYG_ERR_HIP;
        if (sdev != dev) return PYG_ERR_INVALID_ARG;  // the stream must belong to the current device
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PYG_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return PYG_OK;
}

}  // namespace

extern "C" int pyg_propagate_noalloc(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index,
                                     int64_t E, const float *edge_weight, const pyg_csr *csr, int msg, int aggr,
                                     int kernel, void *out, int64_t *argmax, void *stream) {
    // every argument check first (host only), then the scratch the call needs
    size_t need = 0;
    PYG_TRY(pyg::propagate_check(x, dtype, N, F, edge_index, E, edge_weight, csr, msg, aggr, kernel, out, argmax,
                                 &need));
    if (need > kNoallocScratchBytes) return PYG_ERR_UNSUPPORTED;
    void *ws = nullptr;
    PYG_TRY(device_scratch(stream, &ws));
    return pyg_propagate(x, dtype, N, F, edge_index, E, edge_weight, csr, msg, aggr, kernel, out, argmax, ws,
                         kNoallocScratchBytes, stream);
}
