// Device scratch that the library holds for callers that cannot allocate
// (sparse_accumulate_static): one array per device, from the first use of
// the library on that device until the process ends.  Nothing here
// allocates: the array is part of the library's device code object.
#include <mutex>

#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
void *g_scratch[kMaxDevices];   // device address of `scratch` per device; null = not looked up
std::mutex g_scratch_mutex;

}  // namespace

// In host code `scratch` names a host-side stand-in, not device memory: the
// device address comes from the runtime, looked up once per device with that
// device current, and only that address is ever handed to a kernel.
hipError_t static_scratch(void **ptr) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch[dev] == nullptr) {
        void *p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return err;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *ptr = g_scratch[dev];
    return hipSuccess;
}

}  // namespace efs
