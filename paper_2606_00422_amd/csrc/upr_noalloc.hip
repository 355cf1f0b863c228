// Scratch memory of upr_rank_candidates_noalloc: a fixed array in the
// library's device image, so that the call needs no allocation.  Every GPU
// that loads the library holds its own copy at its own address until the
// process ends.
#include <mutex>

#include "upr_internal.h"

// In host code this name is a host-side stand-in, not a device address; the
// device address comes from hipGetSymbolAddress, per device.
static __device__ __attribute__((aligned(256))) unsigned char scratch[UPR_NOALLOC_SCRATCH_BYTES];

namespace upr {

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];      // per device; null until looked up

}  // namespace

hipError_t noalloc_scratch(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_scratch[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr || reinterpret_cast<uintptr_t>(p) % 256 != 0) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *ptr = g_scratch[dev];
    return hipSuccess;
}

}  // namespace upr
