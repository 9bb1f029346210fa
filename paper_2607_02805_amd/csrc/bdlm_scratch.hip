// bdlm_scratch.hip -- the device scratch of the no-allocation prefill
// (bdlm_prefill_noalloc): a file-scope device array the library owns, so the call
// needs no caller workspace and allocates nothing.
//
// Each device the library runs on holds its own copy of the array from the time the
// library's code is loaded there until the process ends.  Host code never passes the
// array's name to a kernel or a copy (on the host that name is a stand-in, not a
// device address): the device address is looked up once per device with
// hipGetSymbolAddress, with that device current, and that pointer is used instead.
// Calls share the array: two calls that overlap on one device race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "bdlm.h"
#include "bdlm_launch.h"

static __device__ __align__(256) unsigned char scratch[BDLM_SCRATCH_BYTES];

namespace bdlm {
namespace {
constexpr int kMaxDevices = 256;
void *g_scratch[kMaxDevices];   // device address of `scratch`, per device ordinal
std::mutex g_scratch_mu;
}  // namespace

int scratch_pointer(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return BDLM_E_LAUNCH;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return BDLM_E_LAUNCH;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return BDLM_OK;
}

}  // namespace bdlm
