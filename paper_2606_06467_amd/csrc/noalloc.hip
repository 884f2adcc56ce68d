// Fixed device scratch of clsa_decode_step_noalloc, the variant of the step for
// callers that cannot allocate (code under graph capture, serving loops,
// harnesses that forbid allocation).  The step's workspace (scores, coarse
// histograms, top-k bitmaps and candidates, split partials) is carved out of a
// file-scope device array instead of a caller buffer.  Every device the
// library runs on holds its own copy of the array until the process ends.
#include <hip/hip_runtime.h>

#include <atomic>

#include "clsa_internal.h"

namespace clsa {

// The array's name is only a host-side stand-in in host code: its device
// address comes from hipGetSymbolAddress, once per device, and only that
// address is ever handed to kernels or copies.
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

static std::atomic<void *> g_scratch_addr[kMaxDevices];

hipError_t noalloc_scratch(void **ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void *p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
        // this device is current: the address of its copy of the array
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_addr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return hipSuccess;
}

}  // namespace clsa
