// Device-resident scratch for the allocation-free decode entry point.
//
// kvp_decode_step_noalloc runs kvp_decode_step's kernels with their workspace (Q, the
// attention output, the residual stream, the split-K partial sums of the projections and
// of the attention) in a file-scope device array instead of a caller buffer, for callers
// that cannot allocate device memory.  Every GPU the library runs on holds one copy of the
// array (kStaticScratchBytes) until the process ends; calls on one GPU share it.
//
// In host code `scratch` names a host-side stand-in for the array, not its device
// address: the address is looked up once per device with hipGetSymbolAddress (with that
// device current) and kept here, and only that address is ever handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.h"

namespace kvp {
namespace {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

hipError_t static_scratch(void** addr, size_t* bytes) {
    *addr = nullptr;
    *bytes = 0;
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
    *bytes = kStaticScratchBytes;
    return hipSuccess;
}

}  // namespace kvp
