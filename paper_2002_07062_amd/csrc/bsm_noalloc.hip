// The statically allocated device buffer behind bsm_softmax_noalloc: each call writes its work
// table here instead of into memory the library allocates, for callers that cannot allocate.
#include <hip/hip_runtime.h>

#include <mutex>

#include "bsm.h"
#include "bsm_launch.hpp"

namespace {

// One copy on every device the library runs on, held until the process ends.  In host code
// this name stands for a host-side shadow, not a device address: the device address of each
// device's copy comes from hipGetSymbolAddress (noalloc_scratch below).
static __device__ __align__(256) unsigned char scratch[BSM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

namespace bsm {

hipError_t noalloc_scratch(int device, void** ptr) {
    *ptr = nullptr;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch_ptr[device]) {
        // the caller has made `device` current: this is its copy's address
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[device] = p;
    }
    *ptr = g_scratch_ptr[device];
    return hipSuccess;
}

}  // namespace bsm
