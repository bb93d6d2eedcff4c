// Decode forward without allocation: the decode kernels' workspace (per-slice
// top-K survivors, per-part records {m, l, s^, o[d]}) lives in a file-scope
// device array instead of a caller-provided buffer, for callers that cannot
// allocate device memory (graph capture, tight serving loops).
//
// Every GPU the library runs on holds its own copy of `scratch` until the
// process ends.  In host code `scratch` names a host-side stand-in, not the
// device array: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and kept, and only that
// address is passed to the kernels.  The decode kernels write every workspace
// byte they later read, so nothing needs clearing between calls; calls that
// overlap on one GPU (two streams, two threads) share the array and race.
#include <mutex>

#include "hils_internal.hpp"

namespace hils {

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

}  // namespace

size_t decode_noalloc_capacity() { return kScratchBytes; }

hipError_t decode_noalloc_scratch(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch[dev] = p;
    }
    *ptr = g_scratch[dev];
    return hipSuccess;
}

}  // namespace hils
