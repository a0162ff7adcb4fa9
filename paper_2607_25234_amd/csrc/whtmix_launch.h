// Internal interface between the C entry points and the kernel launchers.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace whtmix {

enum Dtype { DTYPE_F32 = 0, DTYPE_BF16 = 1 };

// A fully validated call: shapes are powers of two, pointers are non-null
// and aligned, `ws` holds at least B * 2^K floats when plan is THREE_PASS.
struct LaunchArgs {
    const void *x;
    const float *gain;
    void *y;
    float *ws;
    int64_t B;
    int K;          // log2(N * C)
    int dtype;      // Dtype
    int plan;       // PlanKind, resolved (never AUTO)
    hipStream_t stream;
    hipEvent_t events[4];   // optional, may be null
};

// Enqueues the plan's kernels on a.stream.  Returns the first HIP error.
hipError_t launch(const LaunchArgs &a);

}  // namespace whtmix
