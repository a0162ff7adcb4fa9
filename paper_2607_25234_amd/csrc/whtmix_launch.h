// Internal interface between the C entry points and the kernel launchers.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace whtmix {

enum Dtype { DTYPE_F32 = 0, DTYPE_BF16 = 1 };
enum GainKind { GAIN_FULL = 0, GAIN_LOG_SEPARABLE = 1 };

// A fully validated call: C is a power of two, the token axis is padded to
// N_pad = 2^ceil(log2 N), pointers are non-null and aligned, `ws` holds at
// least B * 2^K floats when plan is THREE_PASS.
struct LaunchArgs {
    const void *x;
    void *y;
    int gain_kind;          // GainKind
    const float *gain;      // GAIN_FULL: [N_pad][C]
    const float *gain_t;    // GAIN_LOG_SEPARABLE: [N_pad] log gains over tokens
    const float *gain_c;    //                     [C] log gains over channels
    int cbits;              // log2(C)
    float *ws;
    int64_t B;
    int K;                  // log2(N_pad * C)
    uint32_t nvalid;        // N * C: elements of one slice of x and y
    int dtype;      // Dtype
    int plan;       // PlanKind, resolved (never AUTO)
    hipStream_t stream;
    hipEvent_t events[4];   // optional, may be null
};

// Enqueues the plan's kernels on a.stream.  Returns the first HIP error.
hipError_t launch(const LaunchArgs &a);

}  // namespace whtmix
