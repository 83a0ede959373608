// The fixed device scratch of quarot_linear_e3m2_scratch: the e3m2 codes and
// per-token scales of the activations live in a file-scope device array
// instead of a caller-supplied workspace, for callers that cannot allocate.
//
// Host code never passes the array's name to a kernel or a copy: on the
// host that name is only a stand-in for the symbol.  The device address is
// looked up once per device, with that device current, and kept.
#include <mutex>

#include "../../include/quarot.h"
#include "common.hpp"

namespace quarot {

static __device__ __align__(256) uint8_t scratch[QUAROT_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_ptr[kMaxDevices];  // device address of `scratch` per device, once known

}  // namespace

hipError_t scratch_buffer(void **ptr)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!p)
            return hipErrorInvalidSymbol;
        g_ptr[dev] = p;
    }
    *ptr = g_ptr[dev];
    return hipSuccess;
}

}  // namespace quarot
