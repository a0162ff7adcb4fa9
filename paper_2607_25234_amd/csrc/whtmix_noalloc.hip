// Fixed device scratch for whtmix_forward_noalloc: the float32 workspace of
// the three-pass, two-pass and wave-tile plans in a file-scope device array, so that the call makes
// no allocation (for callers that cannot allocate: code under HIP graph
// capture, tight serving loops).
//
// In host code `scratch` names a host-side stand-in, not device memory; the
// array's device address comes from hipGetSymbolAddress, once per device
// (each device holds its own copy at its own address), and only that
// address is ever passed to kernels.  Every call on a device shares its
// array: calls that overlap on one device race.  Each plan writes every
// workspace element before reading it, so nothing needs clearing.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "whtmix_launch.h"

namespace whtmix {

static __device__ __align__(256) float scratch[kNoAllocScratchFloats];

namespace {
std::mutex g_scratch_mutex;
std::map<int, float *> g_scratch;   // device -> device address of `scratch`
}  // namespace

hipError_t noalloc_scratch(float **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    auto it = g_scratch.find(dev);
    if (it == g_scratch.end()) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        it = g_scratch.emplace(dev, static_cast<float *>(p)).first;
    }
    *out = it->second;
    return hipSuccess;
}

}  // namespace whtmix
