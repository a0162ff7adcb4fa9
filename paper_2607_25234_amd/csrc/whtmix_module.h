// Internal interface between the C entry points and the kernels of the whole
// block with its projections (whtmix_module.hip).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "whtmix_launch.h"
#include "whtmix_plan.h"

namespace whtmix {

// ---------------------------------------------------------------- the block
// How the block with its projections runs (whtmix_module.hip):
//   SMALL       the mixer's SMALL plan, projections on the VALU in LDS;
//   FUSED_MFMA  16 <= C <= 128 with the FUSED or THREE_PASS plan: MFMA
//               prologue and epilogue inside the mixer's kernels;
//   UNFUSED     any other C: projection kernels around the fp32 mixer.
enum ModulePath { MODULE_SMALL = 0, MODULE_FUSED_MFMA = 1, MODULE_UNFUSED = 2 };
constexpr int kModuleMfmaMinCbits = 4;
constexpr int kModuleMfmaMaxCbits = 7;
constexpr int kModuleMaxCbits = 12;   // weights of C*C elements, C <= 4096

inline int module_path(int plan, int cbits)
{
    if (plan == PLAN_SMALL) return MODULE_SMALL;
    if (cbits >= kModuleMfmaMinCbits && cbits <= kModuleMfmaMaxCbits) return MODULE_FUSED_MFMA;
    return MODULE_UNFUSED;
}

// A validated call of the block.  Workspace: the THREE_PASS workspace `ws`
// (B * 2^K floats, else none), then for UNFUSED `z` (B * N * C floats), then
// `wpack` (the two repacked weight matrices; not SMALL).
struct ModuleArgs {
    const void *x;
    const void *w_in;       // [C][C], dtype of x
    const void *w_out;      // [C][C]
    void *y;
    int gain_kind;          // GainKind
    const float *gain;
    const float *gain_t;
    const float *gain_c;
    int cbits;
    float *ws;
    void *wpack;
    float *z;
    int64_t B;
    int K;
    uint32_t nvalid;
    int dtype;
    int plan;
    hipStream_t stream;
    hipEvent_t events[4];   // FUSED_MFMA three-pass: around each of the three
                            // passes; otherwise [0] before, [1] after
};

hipError_t launch_module(const ModuleArgs &m);

}  // namespace whtmix
