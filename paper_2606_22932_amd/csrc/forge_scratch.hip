// forge_scratch.hip -- the library's one fixed device buffer, for the entry point that
// allocates nothing (forge_linear_step_unfused_noalloc): the gradient that the two-kernel
// step materialises between its GEMM and its optimizer kernel lives here instead of in a
// caller-provided workspace.
//
// The array is part of the library's code object, so every device the library runs on
// holds SCRATCH_BYTES of it from the code object's load until the process ends.  In host
// code its name stands for a host-side shadow, not a device address: the device address
// is obtained once per device with hipGetSymbolAddress and only that address is handed to
// kernels.
#include <mutex>

#include "forge_internal.h"

namespace forge_impl {

static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

hipError_t scratch_address(void **out)
{
    static std::mutex mu;
    static void *addr[MAX_DEVICES] = {nullptr};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void *p = nullptr;
        // with `dev` current: the address of this device's copy of the array
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
}

}  // namespace forge_impl
