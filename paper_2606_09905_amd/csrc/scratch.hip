// scratch.hip -- the fixed device scratch of the allocation-free entry
// point.
//
// One array per GPU, reserved when the library's code object is loaded on
// that device and held until the process ends.  In host code the array's
// name is only a host-side handle for the symbol, never a device address:
// its device address is looked up once per device (with that device
// current) and kept; every kernel argument, fill or copy that refers to the
// scratch uses that address.
#include <hip/hip_runtime.h>

#include <mutex>

#include "qx_internal.h"

static __device__ __align__(256) unsigned char scratch[qx::kScratchBytes];

namespace qx {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};
}  // namespace

hipError_t scratch_device_ptr(int dev, void** out) {
    *out = nullptr;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p || ((uintptr_t)p & 255)) return hipErrorInvalidSymbol;
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return hipSuccess;
}

}  // namespace qx
