// svf_noalloc.hip -- device scratch of the no-allocation entry point
// (svf_run_noalloc): one static array per GPU, holding every intermediate
// buffer of a call.
//
// In host code the array's name is only a host-side stand-in; its device
// address is obtained once per device with hipGetSymbolAddress (with that
// device current) and only that address is handed to copies and kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "svf_kernels.h"
#include "svfsim.h"

static __device__ __align__(256) unsigned char scratch[SVF_NOALLOC_SCRATCH_BYTES];

namespace svfk {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices];  // device address of ``scratch`` on each device (null: not yet)

}  // namespace

hipError_t noalloc_scratch(void** addr, size_t* bytes) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_addr[dev] = p;
    }
    *addr = g_addr[dev];
    *bytes = sizeof(scratch);
    return hipSuccess;
}

}  // namespace svfk
