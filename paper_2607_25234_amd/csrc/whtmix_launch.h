// Internal interface between the C entry points and the kernel launchers.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "whtmix_plan.h"

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
    bool pair_outer;        // launch_middle only: the outer passes used 2^16 tiles
    uint32_t *counters;     // ONE_LAUNCH: kCounterWords words, zero between calls
    uint32_t spin_limit;    // ONE_LAUNCH: polls per wait before the call fails
};

// Enqueues the plan's kernels on a.stream.  Returns the first HIP error.
hipError_t launch(const LaunchArgs &a);

// Enqueues the wave-tile kernels (whtmix_wave.hip): a.plan is WAVE_TILES
// (three launches), TWO_PASS (two launches; a.K is 15 or 16) or ONE_LAUNCH
// (one cooperative launch; a.B <= kOneLaunchMaxBatch and a.counters a
// zeroed-or-reset counter block); 12 <= a.K <= 16, a.nvalid a multiple of 8,
// a.ws holding a.B * 2^K floats.
hipError_t launch_wave(const LaunchArgs &a);

// Device address of the fixed scratch array on the current device
// (kNoAllocScratchFloats floats; whtmix_noalloc.hip).  Looks the address up
// once per device; allocates nothing.
hipError_t noalloc_scratch(float **out);

// A validated backward call.  dX = the mixer applied to dY (may be null);
// the gain gradient goes to dgain (joint) or dgt/dgc (separable log gains),
// any of which may be null to skip it.
struct BackwardArgs {
    const void *x;
    const void *dy;
    void *dx;
    int gain_kind;          // GainKind
    const float *gain;
    const float *gain_t;
    const float *gain_c;
    float *dgain;           // [N_pad][C], overwritten
    float *dgt;             // [N_pad], overwritten
    float *dgc;             // [C], overwritten
    int cbits;
    float *ws;              // backward_layout(...).floats floats
    int64_t B;
    int K;
    uint32_t nvalid;
    int dtype;
    int plan;
    hipStream_t stream;
    hipEvent_t events[4];   // [0] before, [1] after the gain gradient, [2] after dX
};

// Workspace plan of a backward call (offsets and sizes in floats).
struct BackwardLayout {
    uint64_t wsx, wsd;      // low-bit transforms of x and dy (three-pass)
    uint64_t part;          // per-chunk partial dG sums (when nchunks > 1)
    uint64_t dg;            // dG for the separable reductions
    uint64_t colpart;       // column partial sums (separable)
    uint64_t rowpart;       // row and column partial sums formed by the middle
    uint64_t fcolpart;      // pass (separable, sep_fused)
    uint32_t nchunks, per_chunk;
    uint32_t rows_per_block, col_blocks;
    uint32_t sep_fused;     // separable: the middle pass forms the partial sums itself
    uint64_t floats;        // total workspace
};

BackwardLayout backward_layout(int plan, int K, int64_t B, int64_t C, bool separable);

hipError_t launch_backward(const BackwardArgs &a);

// Only the middle phase of the three-pass backward (three_pass_split): a.ws
// holds backward_layout's wsx and wsd, the outer forward transforms of x and
// dy made by the caller.  Writes the gain gradient (which must be requested)
// and leaves the mixer of both x and dY up to its last pass in wsx and wsd
// (the middle pass of each, in place).  Slices of 2^12..2^28 elements.
hipError_t launch_backward_middle(const BackwardArgs &a);

// Enqueues only the middle pass of the block's three-pass plan (module_split,
// or pair_split when a.pair_outer; a.ws holds the first outer pass's output);
// a.x, a.y, a.nvalid and a.dtype are not used.
hipError_t launch_middle(const LaunchArgs &a);


}  // namespace whtmix
