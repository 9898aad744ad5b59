// Library-owned device scratch for coded_matmul_noalloc: a file-scope device
// array that every call on a GPU reuses, so that entry point allocates no
// device memory.  Each GPU holds its own copy of the array (from module load
// until the process ends), at its own address.
//
// In host code `scratch` names a host-side stand-in, not a device address;
// the device address is looked up once per device with hipGetSymbolAddress
// (with that device current) and only that address is handed to kernels.
#include <mutex>

#include "internal.h"

namespace coded {
namespace {

static __device__ __align__(256) unsigned char scratch[CODED_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

coded_status static_scratch(void** out) {
    *out = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(CODED_ERR_UNSUPPORTED, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(CODED_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return CODED_OK;
}

}  // namespace coded
