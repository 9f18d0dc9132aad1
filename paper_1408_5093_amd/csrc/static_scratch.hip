// static_scratch.hip -- the library-owned device buffer behind
// caffe_conv_forward_noalloc, the forward entry point for callers that cannot
// allocate device memory.
//
// `scratch` is a file-scope device array: every GPU the library runs on holds
// its own copy, at its own address, from the first use until the process
// ends.  In host code the name `scratch` is only a host-side stand-in for the
// symbol, never a device address; the device address is looked up once per
// device with hipGetSymbolAddress (with that device current) and cached, and
// only that address is ever handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace caffe_hip {

static __device__ __align__(256) char scratch[kStaticScratchBytes];

hipError_t static_scratch_address(void** ptr)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (p == nullptr)
            return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

}  // namespace caffe_hip
