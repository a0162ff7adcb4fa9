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
//   FUSED_MFMA  16 <= C <= 128 with the FUSED or THREE_PASS plan, and bf16
//               C = 256 with the THREE_PASS plan from 2^17 elements per slice
//               (2^16 outer tiles): MFMA prologue and epilogue inside the
//               mixer's kernels;
//   UNFUSED     any other C: projection kernels around the fp32 mixer.
enum ModulePath { MODULE_SMALL = 0, MODULE_FUSED_MFMA = 1, MODULE_UNFUSED = 2 };
constexpr int kModuleMfmaMinCbits = 4;
constexpr int kModuleMfmaMaxCbits = 7;
constexpr int kModuleMaxCbits = 12;   // weights of C*C elements, C <= 4096

inline int module_path(int plan, int cbits, int dtype, int K)
{
    if (plan == PLAN_SMALL) return MODULE_SMALL;
    if (cbits >= kModuleMfmaMinCbits && cbits <= kModuleMfmaMaxCbits) return MODULE_FUSED_MFMA;
    if (cbits == kPairModuleCbits && dtype == DTYPE_BF16 && plan == PLAN_THREE_PASS &&
        K >= kPairModuleMinK)
        return MODULE_FUSED_MFMA;
    return MODULE_UNFUSED;
}

// Flat-index bits of the outer passes of the block's THREE_PASS plan.
inline int module_outer_bits(int path, int cbits, int K)
{
    if (path == MODULE_FUSED_MFMA)
        return cbits == kPairModuleCbits ? pair_split(K).A : module_split(K).A;
    return three_pass_split(K).A;   // UNFUSED: the mixer's own plan
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

// ---------------------------------------------------------------- backward
// Split of a weight gradient dW = A^T B over rows (A, B [rows][C]): `chunks`
// partial C x C sums of `rows_per_chunk` rows each, added in a fixed order:
// first in groups of kWgradGroup consecutive chunks, then the group sums.
constexpr uint32_t kWgradGroup = 16;
struct WgradPlan {
    uint32_t chunks;
    uint32_t rows_per_chunk;
    uint32_t groups() const { return (chunks + kWgradGroup - 1) / kWgradGroup; }
    // floats of partial sums: the chunks' and the groups'
    uint64_t partial_floats(int cbits) const
    {
        return (uint64_t)(chunks + groups()) << (2 * cbits);
    }
};

// About 512 workgroups (two per CU) over the chunks and the (C/T)^2 output
// blocks of the matrix-core kernel (T = min(C, 128)), at least 64 rows per
// chunk; C < 16 (the VALU kernel, one block per chunk) the same.
inline WgradPlan wgrad_plan(uint64_t rows, int cbits)
{
    if (rows == 0) return WgradPlan{0, 4};   // no partials: the sums are zero
    const uint64_t C = uint64_t(1) << cbits;
    const uint64_t T = C < 128 ? C : 128;
    const uint64_t blocks = C >= 16 ? (C / T) * (C / T) : 1;
    uint64_t chunks = 512 / blocks;
    if (chunks < 1) chunks = 1;
    const uint64_t most = (rows + 63) / 64;   // at least 64 rows per chunk
    if (chunks > most) chunks = most;
    uint64_t rpc = (rows + chunks - 1) / chunks;
    rpc = (rpc + 3) / 4 * 4;
    if (rpc == 0) rpc = 4;
    return WgradPlan{(uint32_t)((rows + rpc - 1) / rpc), (uint32_t)rpc};
}

// The block's backward runs its projections inside the mixer backward's
// passes (THREE_PASS, when a gain gradient is requested: 16 <= C <= 128 on
// slices up to 2^25 elements, and bf16 C = 256 on 2^26..2^28, where the
// block's and the mixer's splits agree); otherwise as projection kernels
// around the mixer's forward and backward on float32 Z, Z' and dZ'.
inline bool module_backward_fused(int plan, int cbits, int dtype, int K)
{
    if (plan != PLAN_THREE_PASS) return false;
    if (cbits >= kModuleMfmaMinCbits && cbits <= kModuleMfmaMaxCbits) return K >= 12 && K <= 25;
    return dtype == DTYPE_BF16 && cbits == kPairModuleCbits && K >= 26 && K <= 28;
}

// A validated backward call of the block.  Workspace pieces (floats unless
// noted): z, zp, dzp [B*N*C] (Z = X W_in, Z' = mixer(Z), dZ' then dZ);
// wpack: W_in, W_out^T and W_in^T packed (3*C*C elements of the dtype);
// wpart: wgrad_plan(B*N, cbits).chunks * C*C partial sums; mix_ws: the
// THREE_PASS workspace (B * 2^K, else none); bwd_ws: the mixer backward's
// workspace (backward_layout).
struct ModuleBackwardArgs {
    const void *x;
    const void *w_in;
    const void *w_out;
    const void *dy;
    void *dx;               // [B][N][C] dtype
    float *dw_in;           // [C][C]
    float *dw_out;          // [C][C]
    int gain_kind;
    const float *gain;
    const float *gain_t;
    const float *gain_c;
    float *dgain;
    float *dgt;
    float *dgc;
    int cbits;
    int64_t B;
    int K;
    uint32_t nvalid;        // N * C
    int dtype;
    int plan;               // the mixer's plan for [B, N, C]
    hipStream_t stream;
    hipEvent_t events[4];   // [0] before; then after each phase: unfused, [1] Z, Z',
                            // dZ', dW_out, [2] the mixer's gradient, [3] dX and dW_in;
                            // fused, [1] the transforms of Z and dZ' and dG, [2] Z'
                            // and dW_out, [3] dX and dW_in
    float *z;
    float *zp;
    float *dzp;
    void *wpack;
    float *wpart;
    float *mix_ws;
    float *bwd_ws;
};

hipError_t launch_module_backward(const ModuleBackwardArgs &m);

}  // namespace whtmix
