// Fixed device scratch for alp_search_batch_async_noalloc: one array per GPU, holding every
// buffer a search launch needs beyond its inputs and outputs, so that the entry point allocates
// nothing.
//
// In host code `scratch` is only a host-side stand-in for the device array: its device address
// comes from hipGetSymbolAddress, taken once per device with that device current (by
// alp_load_profiles, the library's set-up call) and kept per device.  Host code passes that
// address, never the array's name, to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "alp.h"
#include "alp_internal.h"

namespace {

static __device__ __align__(256) uint8_t scratch[ALP_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

std::mutex g_mutex;
bool g_looked_up[kMaxDevices] = {};
void *g_address[kMaxDevices] = {};
hipError_t g_status[kMaxDevices] = {};

}  // namespace

namespace alp {

hipError_t static_scratch_address(int device, void **ptr)
{
    *ptr = nullptr;
    if (device < 0 || device >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mutex);
    if (!g_looked_up[device]) {
        // The caller makes `device` current first: each GPU holds its own copy of the array.
        int current = -1;
        hipError_t e = hipGetDevice(&current);
        if (e != hipSuccess)
            return e;
        if (current != device)
            return hipErrorInvalidDevice;
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_status[device] = e;
        g_address[device] = e == hipSuccess ? p : nullptr;
        g_looked_up[device] = true;
    }
    *ptr = g_address[device];
    return g_status[device];
}

}  // namespace alp
