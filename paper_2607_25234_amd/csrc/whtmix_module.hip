// The whole WHTMix block (section III-B, eqs. (1)-(4)) for gfx950:
//     Z = X W_in;   Z <- mixer(Z);   Y = Z W_out
// with the projections fused into the mixer's first and last kernels as an
// MFMA prologue and epilogue, so Z never makes an extra trip through HBM.
//
// Projections (C = 2^CB channels, 16 <= C <= 128):
//   * bf16: v_mfma_f32_16x16x32_bf16 (v_mfma_f32_16x16x16_bf16 for C = 16).
//     X W_in multiplies bf16 by bf16, which is exact in the fp32 accumulator.
//     Z' W_out has an fp32 left operand: it is split as Z' = hi + lo (two
//     bf16, hi = RNE(Z'), lo = RNE(Z' - hi), which leaves a residual below
//     2^-17 |Z'|) and multiplied in two MFMAs.
//   * fp32: v_mfma_f32_16x16x4_f32.
//   The contraction order over k is free, so each lane's k values are chosen
//   to make its loads of X 16-byte pieces and its register reads contiguous.
//
// Register layouts (whtmix_tile.h defines "layout S").  With the lane layout of
// the 16x16 MFMA result (lane = 16*q + j holds rows 4q + r, r = 0..3, of
// column j), the fragments of Z = X W_in for a wave's 16*2^(7-CB) tokens are
// exactly layout 4 (registers hold tile bits [4, 9)) after a renumbering of
// registers, for every C in [16, 128]: the prologue feeds the transform with
// no extra LDS pass.  The epilogue computes Y^T = W_out^T Z'^T, whose right
// operand wants lane j on a token and lanes q on channel groups; the last
// inverse exchange delivers that "epilogue layout" directly (Epi below).
// The weights are repacked once per call into the MFMA operand order, staged
// whole into LDS by each workgroup and read as one 8- or 16-byte LDS load per
// lane per MFMA.
//
// Plans (the mixer's, whtmix_plan.h):
//   FUSED       K <= 15: one workgroup per slice, prologue + mixer + epilogue.
//   THREE_PASS  prologue in the first outer pass, the unchanged middle pass,
//               epilogue in the second outer pass; bf16 C = 256 on 2^16
//               outer tiles of two register sets (the pair kernels below).
//   SMALL       K <= 10: one LDS-resident workgroup per slice, VALU products.
//   UNFUSED     any other shape: projection kernels around the fp32 mixer (on
//               the matrix cores from C = 256 where a weight slice fits LDS).
// The block's backward fuses its projections into the mixer backward's
// passes for bf16 32 <= C <= 128 (module_backward_fused_k).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "whtmix_launch.h"
#include "whtmix_module.h"
#include "whtmix_plan.h"
#include "whtmix_tile.h"

namespace whtmix {
namespace {

using namespace tile;

typedef short bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- layouts
// A layout names the tile bit held by each register bit (reg) and the tile
// index of a thread's register 0 (base).  Register offsets and LDS offsets
// pad() are additive over the disjoint bit fields, as in whtmix_tile.h.
template <int S>
struct Std {
    static constexpr int reg(int j) { return S + j; }
    __device__ static uint32_t base(uint32_t tau) { return layout_base<S>(tau); }
};

// Epilogue layout of a 2^M tile with C = 2^CB (flat t = token * C + channel):
//   lanes 0-3  -> token bits 0-3           (the MFMA column j)
//   lanes 4-5  -> channel bits CB-2, CB-1  (the MFMA k group q)
//   waves      -> token bits 4 .. M-8
//   registers  -> channel bits 0 .. CB-3, then token bits M-7 .. M-CB-1
// so a lane holds C/4 consecutive channels of 2^(7-CB) tokens.
template <int M, int CB>
struct Epi {
    static constexpr int reg(int j) { return j < CB - 2 ? j : M - 7 + CB + (j - (CB - 2)); }
    __device__ static uint32_t base(uint32_t tau)
    {
        return ((tau & 15u) << CB) | (((tau >> 4) & 3u) << (CB - 2)) | ((tau >> 6) << (CB + 4));
    }
};

// 2^15 tiles: registers hold t bits 0-3 and 9; threads hold bits 4-8
// (lanes 0-4) and 10-14.  From layout 4, where bits 4-8 are done, one
// exchange reaches every bit below 10.
struct Low4Hi9 {
    static constexpr int reg(int j) { return j < 4 ? j : 9; }
    __device__ static uint32_t base(uint32_t tau) { return ((tau & 31u) << 4) | ((tau >> 5) << 10); }
};

template <class L>
constexpr uint32_t reg_offset(uint32_t k)
{
    uint32_t t = 0;
    for (int j = 0; j < VB; ++j)
        if (k & (1u << j)) t |= 1u << L::reg(j);
    return t;
}

// Re-lay the tile from LA to LB through LDS (LEAD: wait for the previous
// readers of the LDS first).
template <class LA, class LB, bool LEAD = true>
__device__ __forceinline__ void relayout(float *lds, float (&v)[V], uint32_t tau)
{
    const uint32_t pa = pad(LA::base(tau));
    const uint32_t pb = pad(LB::base(tau));
    if (LEAD)
        __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pa + pad(reg_offset<LA>((uint32_t)k))] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        v[k] = lds[pb + pad(reg_offset<LB>((uint32_t)k))];
}

// Butterflies over the register bits set in MASK.
template <uint32_t MASK>
__device__ __forceinline__ void butterflies_on(float (&v)[V])
{
#pragma unroll
    for (int j = 0; j < VB; ++j) {
        if (!(MASK & (1u << j))) continue;
#pragma unroll
        for (int k = 0; k < V; ++k) {
            if (!(k & (1 << j))) {
                const float a = v[k];
                const float b = v[k | (1 << j)];
                v[k] = a + b;
                v[k | (1 << j)] = a - b;
            }
        }
    }
}

// Forward transform of a 2^M tile arriving in layout 4 from the prologue
// (bits [4, 9) still to do): ends in layout M-5 with every bit done.
template <int M>
__device__ __forceinline__ void forward_from_prologue(float *lds, float (&v)[V], uint32_t tau)
{
    butterflies_on<31>(v);
    // LEAD: the weights (or the previous register set) were read from LDS
    if constexpr (M <= 14) {
        relayout<Std<4>, Std<0>, true>(lds, v, tau);
        butterflies_on<15>(v);                      // bits 0-3
        relayout<Std<0>, Std<M - 5>>(lds, v, tau);
        butterflies_on<31u & ~((1u << (14 - M)) - 1u)>(v);   // bits 9 .. M-1
    } else {
        relayout<Std<4>, Low4Hi9, true>(lds, v, tau);
        butterflies_on<31>(v);                      // bits 0-3 and 9
        relayout<Low4Hi9, Std<10>>(lds, v, tau);
        butterflies_on<31>(v);                      // bits 10-14
    }
}

// Inverse transform of a 2^M tile in layout M-5 (nothing done yet), ending
// in the epilogue layout with every bit done.  The epilogue layout's register
// bits are left to the last step; the others go first.
template <int M, int CB, bool LEAD0>
__device__ __forceinline__ void inverse_to_epilogue(float *lds, float (&v)[V], uint32_t tau)
{
    constexpr int len = M - 3 - CB;   // bits [CB-2, M-5) between the two
    butterflies_on<(1u << (CB - 2)) - 1u>(v);   // bits [M-5, M-7+CB)
    if constexpr (len <= VB) {
        relayout<Std<M - 5>, Std<CB - 2>, LEAD0>(lds, v, tau);
        butterflies_on<(1u << len) - 1u>(v);
        relayout<Std<CB - 2>, Epi<M, CB>>(lds, v, tau);
    } else {
        relayout<Std<M - 5>, Std<CB - 2>, LEAD0>(lds, v, tau);
        butterflies_on<31>(v);
        relayout<Std<CB - 2>, Std<CB + 3>>(lds, v, tau);
        butterflies_on<(1u << (len - VB)) - 1u>(v);
        relayout<Std<CB + 3>, Epi<M, CB>>(lds, v, tau);
    }
    butterflies_on<31>(v);
}

// ---------------------------------------------------------------- projections
template <typename T, int CB>
struct Proj {
    static constexpr int C = 1 << CB;
    static constexpr int NRB = 1 << (7 - CB);    // 16-row MFMA blocks per wave
    static constexpr int NNB = C / 16;           // 16-column blocks
    static constexpr bool BF = sizeof(T) == 2;
    // bf16 from C = 32: the 16x16x32 instruction, KS2 steps of 32 k values
    static constexpr bool X32 = BF && C >= 32;
    static constexpr int KS2 = C / 32;
    // k steps per column block of the 16x16x16 (bf16, C = 16) and 16x16x4
    // (fp32) instructions: 16 or 4 k values per MFMA
    static constexpr int KS = BF ? C / 16 : C / 4;
    // A-fragment registers per lane and row block (X: C/4 values)
    static constexpr uint32_t WBYTES = (uint32_t)C * C * sizeof(T);
};

// k value order of the 16x16x16 bf16 and 16x16x4 fp32 products (the fused
// kernels' float32 and C = 16 forms, and the projection kernel; the fused bf16
// forms from C = 32 use pack_x32_kernel's order).  bf16: lane group q, step
// kk, element r: channel 32(kk/2) + 8q + 4(kk%2) + r (C >= 32; each lane reads
// its channels as 16-byte pieces of 8), or 4q + r (C = 16).  fp32: step s:
// channel 16(s/4) + 4q + s%4 (16-byte pieces of 4).
__host__ __device__ constexpr uint32_t k_in_bf16(uint32_t C, uint32_t kk, uint32_t q, uint32_t r)
{
    return C >= 32 ? 32u * (kk >> 1) + 8u * q + 4u * (kk & 1u) + r : 4u * q + r;
}
__host__ __device__ constexpr uint32_t k_in_f32(uint32_t s, uint32_t q)
{
    return 16u * (s >> 2) + 4u * q + (s & 3u);
}
// Epilogue: lane group q holds channels [q C/4, (q+1) C/4); step kk element r
// (bf16) or step s (fp32) is channel q C/4 + 4 kk + r, or q C/4 + s.
// Output channel of MFMA row m in column block nb: bf16 pairs of blocks give
// each lane 8 consecutive channels (one 16-byte store); fp32 rows are
// 16 nb + m (4 consecutive channels per lane, 16 bytes).
__host__ __device__ constexpr uint32_t oc_bf16(uint32_t C, uint32_t nb, uint32_t m)
{
    return C >= 32 ? 32u * (nb >> 1) + 8u * (m >> 2) + 4u * (nb & 1u) + (m & 3u) : m;
}

// One thread per packed element.  Packed index = ((nb * KS + kk) * 64 + lane)
// * 4 + r with lane = 16 q + j (bf16), or ((nb * C/16 + p) * 64 + lane) * 4 + e
// with step s = 4p + e (fp32).  W_in feeds the B operand of Z = X W_in
// (column 16 nb + j); W_out feeds the A operand of Y^T = W_out^T Z'^T, or
// (out_as_in) the B operand of Y = Z' W_out like W_in.
template <typename T>
__global__ void __launch_bounds__(256)
pack_weights_kernel(const T *__restrict__ w_in, const T *__restrict__ w_out, T *__restrict__ p_in,
                    T *__restrict__ p_out, int cb, int out_as_in)
{
    const uint32_t C = 1u << cb;
    const uint32_t idx = blockIdx.x * 256u + threadIdx.x;
    if (idx >= C * C) return;
    const uint32_t e = idx & 3u;
    const uint32_t lane = (idx >> 2) & 63u;
    const uint32_t j = lane & 15u, q = lane >> 4;
    const uint32_t rest = idx >> 8;
    if constexpr (sizeof(T) == 2) {
        const uint32_t ks = C / 16u;
        const uint32_t kk = rest % ks, nb = rest / ks;
        const uint32_t src = k_in_bf16(C, kk, q, e) * C + 16u * nb + j;
        p_in[idx] = w_in[src];
        p_out[idx] = out_as_in ? w_out[src]
                               : w_out[(q * (C / 4u) + 4u * kk + e) * C + oc_bf16(C, nb, j)];
    } else {
        const uint32_t np = C / 16u;
        const uint32_t p = rest % np, nb = rest / np;
        const uint32_t s = 4u * p + e;
        const uint32_t src = k_in_f32(s, q) * C + 16u * nb + j;
        p_in[idx] = w_in[src];
        p_out[idx] = out_as_in ? w_out[src] : w_out[(q * (C / 4u) + s) * C + 16u * nb + j];
    }
}

// bf16, C >= 32: the operands of v_mfma_f32_16x16x32_bf16, whose lane 16 g + i
// supplies k = 8 g + [0, 8) of row i of A / column i of B.  One thread per
// packed element: index ((nb * C/32 + kk) * 64 + 16 g + j) * 8 + e holds
// W_in[32 kk + 8 g + e][16 nb + j] (B operand of Z = X W_in: step kk of lane
// group g is channels 32 kk + 8 g + [0, 8) of x, one 16-byte load) and
// W_out[(C/4) g + 8 kk + e][oc_bf16(C, nb, j)] (A operand of Y^T = W_out^T Z'^T:
// lane group g holds channels [g C/4, (g+1) C/4) of Z').  The block's backward
// packs transposed matrices in the same orders (dZ' = dY W_out^T through the
// prologue, dX = dZ W_in^T through the epilogue).
enum PackMode { PACK_PROLOGUE = 0, PACK_EPILOGUE = 1, PACK_PROLOGUE_T = 2, PACK_EPILOGUE_T = 3 };

__device__ __forceinline__ uint32_t pack_x32_source(uint32_t idx, uint32_t C, int mode)
{
    const uint32_t e = idx & 7u, lane = (idx >> 3) & 63u;
    const uint32_t j = lane & 15u, g = lane >> 4;
    const uint32_t ks = C / 32u;
    const uint32_t kk = (idx >> 9) % ks, nb = (idx >> 9) / ks;
    // (k, column) of the operand, then the element of W (or of W^T)
    const bool pro = mode == PACK_PROLOGUE || mode == PACK_PROLOGUE_T;
    const uint32_t k = pro ? 32u * kk + 8u * g + e : (C / 4u) * g + 8u * kk + e;
    const uint32_t col = pro ? 16u * nb + j : oc_bf16(C, nb, j);
    return mode >= PACK_PROLOGUE_T ? col * C + k : k * C + col;
}

// Up to three packings in one launch: p[i] = w[i] packed in mode[i] for the
// entries whose p[i] is not null.
template <typename T>
struct PackJobs {
    const T *w[3];
    T *p[3];
    int mode[3];
};
using PackX32Jobs = PackJobs<__bf16>;

__global__ void __launch_bounds__(256)
pack_x32_kernel(PackX32Jobs jobs, int cb)
{
    const uint32_t C = 1u << cb;
    const uint32_t idx = blockIdx.x * 256u + threadIdx.x;
    if (idx >= C * C) return;
#pragma unroll
    for (int i = 0; i < 3; ++i)
        if (jobs.p[i])
            jobs.p[i][idx] = jobs.w[i][pack_x32_source(idx, C, jobs.mode[i])];
}

// The orders of pack_weights_kernel (the 16x16x16 bf16 products at C = 16 and
// the 16x16x4 float32 ones) in the four modes of pack_x32_kernel.
template <typename T>
__device__ __forceinline__ uint32_t pack_std_source(uint32_t idx, uint32_t C, int mode)
{
    const uint32_t e = idx & 3u, lane = (idx >> 2) & 63u;
    const uint32_t j = lane & 15u, q = lane >> 4;
    const uint32_t rest = idx >> 8;
    const bool pro = mode == PACK_PROLOGUE || mode == PACK_PROLOGUE_T;
    uint32_t k, col;
    if constexpr (sizeof(T) == 2) {
        const uint32_t ks = C / 16u, kk = rest % ks, nb = rest / ks;
        k = pro ? k_in_bf16(C, kk, q, e) : q * (C / 4u) + 4u * kk + e;
        col = pro ? 16u * nb + j : oc_bf16(C, nb, j);
    } else {
        const uint32_t np = C / 16u, p = rest % np, nb = rest / np, s = 4u * p + e;
        k = pro ? k_in_f32(s, q) : q * (C / 4u) + s;
        col = 16u * nb + j;
    }
    return mode >= PACK_PROLOGUE_T ? col * C + k : k * C + col;
}

template <typename T>
__global__ void __launch_bounds__(256)
pack_std_kernel(PackJobs<T> jobs, int cb)
{
    const uint32_t C = 1u << cb;
    const uint32_t idx = blockIdx.x * 256u + threadIdx.x;
    if (idx >= C * C) return;
#pragma unroll
    for (int i = 0; i < 3; ++i)
        if (jobs.p[i])
            jobs.p[i][idx] = jobs.w[i][pack_std_source<T>(idx, C, jobs.mode[i])];
}

// X fragments of the prologue: per row block, the lane's C/4 channels of its
// token, as bf16x4 per k step (bf16) or floats (fp32).
template <typename T, int CB>
struct XFrag;

template <int CB>
struct XFrag<__bf16, CB> {
    using P = Proj<__bf16, CB>;
    using Frag = typename std::conditional<P::X32, bf16x8, bf16x4>::type;
    Frag a[P::NRB][P::X32 ? P::KS2 : P::KS];
};
template <int CB>
struct XFrag<float, CB> {
    using P = Proj<float, CB>;
    float a[P::NRB][P::KS];
};

// Token (tile row) of MFMA row m in row block rb for wave w: layout 4 puts
// token bits 0-1 on r = m%4, bits 2 .. 8-CB on rb, the next two on the lane
// group q = m/4 and the rest on the wave.
template <int CB>
__device__ __forceinline__ uint32_t prologue_token(uint32_t rb, uint32_t m, uint32_t w)
{
    return (m & 3u) | (rb << 2) | ((m >> 2) << (9 - CB)) | (w << (11 - CB));
}

// Loads the lane's X fragments from a tile of `valid` elements (a multiple of
// C); rows past it read as zero.  Rows are masked explicitly (the range check
// of a buffer access is not relied on: part of each offset is in soffset).
template <typename T, int CB>
__device__ __forceinline__ void load_x_frags(XFrag<T, CB> &f, const T *tile, uint32_t valid,
                                             bool whole, uint32_t tau)
{
    using P = Proj<T, CB>;
    const uint32_t lane = tau & 63u, w = tau >> 6;
    const uint32_t i = lane & 15u, q = lane >> 4;
    const __amdgpu_buffer_rsrc_t r = buffer(tile, valid * (uint32_t)sizeof(T));
    const uint32_t tok0 = prologue_token<CB>(0, i, w);
    const uint32_t row = tok0 * (uint32_t)(P::C * sizeof(T));
    constexpr uint32_t rb_bytes = 4u * P::C * sizeof(T);
#pragma unroll
    for (int rb = 0; rb < P::NRB; ++rb) {
        const bool ok = whole || (tok0 + 4u * rb) * (uint32_t)P::C < valid;
        if constexpr (P::BF) {
            if constexpr (P::C >= 32) {
#pragma unroll
                for (int p = 0; p < P::C / 32; ++p) {   // channels 32 p + 8 q + [0, 8)
                    u32x4 d = {0u, 0u, 0u, 0u};
                    if (ok)
                        d = __builtin_amdgcn_raw_buffer_load_b128(r, row + 16u * q,
                                                                  rb * rb_bytes + 64u * p,
                                                                  kStreaming);
                    f.a[rb][p] = __builtin_bit_cast(bf16x8, d);
                }
            } else {
                u32x2 d = {0u, 0u};
                if (ok)
                    d = __builtin_amdgcn_raw_buffer_load_b64(r, row + 8u * q, rb * rb_bytes,
                                                             kStreaming);
                f.a[rb][0] = __builtin_bit_cast(bf16x4, d);
            }
        } else {
#pragma unroll
            for (int p = 0; p < P::C / 16; ++p) {
                u32x4 d = {0u, 0u, 0u, 0u};
                if (ok)
                    d = __builtin_amdgcn_raw_buffer_load_b128(r, row + 16u * q,
                                                              rb * rb_bytes + 64u * p,
                                                              kStreaming);
                // Cast the whole vector: this compiler reads element 0 for a
                // __builtin_bit_cast of a single ext-vector element (d.y etc.).
                const f32x4 fv = __builtin_bit_cast(f32x4, d);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    f.a[rb][4 * p + e] = fv[e];
            }
        }
    }
}

// Z = X W_in for the wave's tokens, into v in layout 4: register
// nb | r << (CB-4) | rb << (CB-2) holds tile bits [4, 9) = channel bits 4..CB-1
// (nb), token bits 0-1 (r), token bits 2..8-CB (rb).  wl: packed W_in in LDS.
template <typename T, int CB>
__device__ __forceinline__ void project_in(float (&v)[V], const XFrag<T, CB> &f, const void *wl,
                                           uint32_t tau)
{
    using P = Proj<T, CB>;
    const uint32_t lane = tau & 63u;
    if constexpr (P::X32) {
        const bf16x8 *wb = static_cast<const bf16x8 *>(wl);
#pragma unroll
        for (int nb = 0; nb < P::NNB; ++nb) {
            bf16x8 b[P::KS2];
#pragma unroll
            for (int kk = 0; kk < P::KS2; ++kk)
                b[kk] = wb[(nb * P::KS2 + kk) * 64 + lane];
#pragma unroll
            for (int rb = 0; rb < P::NRB; ++rb) {
                f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int kk = 0; kk < P::KS2; ++kk)
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[rb][kk], b[kk], acc, 0, 0, 0);
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    v[nb | (r << (CB - 4)) | (rb << (CB - 2))] = acc[r];
            }
        }
    } else if constexpr (P::BF) {
        const bf16x4 *wb = static_cast<const bf16x4 *>(wl);
#pragma unroll
        for (int nb = 0; nb < P::NNB; ++nb) {
            bf16x4 b[P::KS];
#pragma unroll
            for (int kk = 0; kk < P::KS; ++kk)
                b[kk] = wb[(nb * P::KS + kk) * 64 + lane];
#pragma unroll
            for (int rb = 0; rb < P::NRB; ++rb) {
                f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int kk = 0; kk < P::KS; ++kk)
                    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(f.a[rb][kk], b[kk], acc, 0, 0,
                                                                     0);
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    v[nb | (r << (CB - 4)) | (rb << (CB - 2))] = acc[r];
            }
        }
    } else {
        const f32x4 *wf = static_cast<const f32x4 *>(wl);
        constexpr int NP = P::C / 16;
#pragma unroll
        for (int nb = 0; nb < P::NNB; ++nb) {
            f32x4 acc[P::NRB];
#pragma unroll
            for (int rb = 0; rb < P::NRB; ++rb)
                acc[rb] = (f32x4){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                const f32x4 b = wf[(nb * NP + p) * 64 + lane];
#pragma unroll
                for (int rb = 0; rb < P::NRB; ++rb) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.a[rb][4 * p + e], b[e],
                                                                       acc[rb], 0, 0, 0);
                }
            }
#pragma unroll
            for (int rb = 0; rb < P::NRB; ++rb)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    v[nb | (r << (CB - 4)) | (rb << (CB - 2))] = acc[rb][r];
        }
    }
}

// Cache policy of the epilogue's y stores.  Each 128-byte line of y is
// written in 64-byte halves by two store instructions (a lane group covers 4
// lanes x 16 bytes of a row); with the non-temporal policy the halves reached
// memory as separate partial writes (1.4x the y bytes in WRITE_SIZE), while
// temporal stores let L2 merge them (exactly the y bytes; 3.9 us faster on
// the stereo64k block, of which the middle pass gives back 2).
constexpr int kYPolicy = kTemporal;

__device__ __forceinline__ uint32_t pack2_bf16(float a, float b)
{
    return (uint32_t)__builtin_bit_cast(unsigned short, (__bf16)a) |
           ((uint32_t)__builtin_bit_cast(unsigned short, (__bf16)b) << 16);
}

// Y = Z' W_out for the wave's tokens, Z' in the epilogue layout of a 2^M
// tile; stores the rows of the tile with element index < valid (a multiple
// of C), masked explicitly.  wl: packed W_out in LDS.
template <typename T, int CB, int M>
__device__ __forceinline__ void project_out(const float (&v)[V], const void *wl, T *tile,
                                            uint32_t valid, uint32_t tau)
{
    using P = Proj<T, CB>;
    const uint32_t lane = tau & 63u, w = tau >> 6;
    const uint32_t j = lane & 15u, q = lane >> 4;
    const __amdgpu_buffer_rsrc_t r = buffer(tile, valid * (uint32_t)sizeof(T));
    const bool whole = valid >= (1u << M);
    // token of column j in row block rb: j | w << 4 | rb << (M-7)
    const uint32_t tok0 = j | (w << 4);
    const uint32_t row = tok0 * (uint32_t)(P::C * sizeof(T));
    constexpr uint32_t rb_bytes = (1u << (M - 7)) * P::C * sizeof(T);
    constexpr int RB_SHIFT = CB - 2;   // register bits of the row block
    if constexpr (P::X32) {
        const bf16x8 *wb = static_cast<const bf16x8 *>(wl);
#pragma unroll
        for (int rb = 0; rb < P::NRB; ++rb) {
            // step kk element e: channel q C/4 + 8 kk + e
            bf16x8 hi[P::KS2], lo[P::KS2];
#pragma unroll
            for (int kk = 0; kk < P::KS2; ++kk) {
                u32x4 h2, l2;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float z0 = v[(8 * kk + 2 * e) | (rb << RB_SHIFT)];
                    const float z1 = v[(8 * kk + 2 * e + 1) | (rb << RB_SHIFT)];
                    const float h0 = (float)(__bf16)z0, h1 = (float)(__bf16)z1;
                    h2[e] = pack2_bf16(z0, z1);
                    l2[e] = pack2_bf16(z0 - h0, z1 - h1);
                }
                hi[kk] = __builtin_bit_cast(bf16x8, h2);
                lo[kk] = __builtin_bit_cast(bf16x8, l2);
            }
            f32x4 acc[P::NNB];
#pragma unroll
            for (int nb = 0; nb < P::NNB; ++nb) {
                acc[nb] = (f32x4){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int kk = 0; kk < P::KS2; ++kk) {
                    const bf16x8 a = wb[(nb * P::KS2 + kk) * 64 + lane];
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, hi[kk], acc[nb], 0, 0, 0);
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, lo[kk], acc[nb], 0, 0, 0);
                }
            }
            // the row block's token; MFMAs above run with every lane active
            const bool ok = whole || (tok0 + ((uint32_t)rb << (M - 7))) * (uint32_t)P::C < valid;
            // blocks 2n, 2n+1: channels 32 n + 8 q + [0, 8)
#pragma unroll
            for (int n = 0; n < P::NNB / 2; ++n) {
                const u32x4 d = {pack2_bf16(acc[2 * n][0], acc[2 * n][1]),
                                 pack2_bf16(acc[2 * n][2], acc[2 * n][3]),
                                 pack2_bf16(acc[2 * n + 1][0], acc[2 * n + 1][1]),
                                 pack2_bf16(acc[2 * n + 1][2], acc[2 * n + 1][3])};
                if (ok)
                    __builtin_amdgcn_raw_buffer_store_b128(d, r, row + 16u * q,
                                                           rb * rb_bytes + 64u * n, kYPolicy);
            }
        }
    } else if constexpr (P::BF) {
        const bf16x4 *wb = static_cast<const bf16x4 *>(wl);
#pragma unroll
        for (int rb = 0; rb < P::NRB; ++rb) {
            bf16x4 hi[P::KS], lo[P::KS];
#pragma unroll
            for (int kk = 0; kk < P::KS; ++kk) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float z = v[(4 * kk + e) | (rb << RB_SHIFT)];
                    const __bf16 h = (__bf16)z;
                    hi[kk][e] = __builtin_bit_cast(short, h);
                    lo[kk][e] = __builtin_bit_cast(short, (__bf16)(z - (float)h));
                }
            }
            f32x4 acc[P::NNB];
#pragma unroll
            for (int nb = 0; nb < P::NNB; ++nb) {
                acc[nb] = (f32x4){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int kk = 0; kk < P::KS; ++kk) {
                    const bf16x4 a = wb[(nb * P::KS + kk) * 64 + lane];
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, hi[kk], acc[nb], 0, 0,
                                                                         0);
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, lo[kk], acc[nb], 0, 0,
                                                                         0);
                }
            }
            // the row block's token; MFMAs above run with every lane active
            const bool ok = whole || (tok0 + ((uint32_t)rb << (M - 7))) * (uint32_t)P::C < valid;
            if constexpr (P::C >= 32) {
                // blocks 2n, 2n+1: channels 32 n + 8 q + [0, 8)
#pragma unroll
                for (int n = 0; n < P::NNB / 2; ++n) {
                    const u32x4 d = {pack2_bf16(acc[2 * n][0], acc[2 * n][1]),
                                     pack2_bf16(acc[2 * n][2], acc[2 * n][3]),
                                     pack2_bf16(acc[2 * n + 1][0], acc[2 * n + 1][1]),
                                     pack2_bf16(acc[2 * n + 1][2], acc[2 * n + 1][3])};
                    if (ok)
                        __builtin_amdgcn_raw_buffer_store_b128(d, r, row + 16u * q,
                                                               rb * rb_bytes + 64u * n,
                                                               kYPolicy);
                }
            } else {
                const u32x2 d = {pack2_bf16(acc[0][0], acc[0][1]),
                                 pack2_bf16(acc[0][2], acc[0][3])};
                if (ok)
                    __builtin_amdgcn_raw_buffer_store_b64(d, r, row + 8u * q, rb * rb_bytes,
                                                          kYPolicy);
            }
        }
    } else {
        const f32x4 *wf = static_cast<const f32x4 *>(wl);
        constexpr int NP = P::C / 16;
#pragma unroll
        for (int rb = 0; rb < P::NRB; ++rb) {
            const bool ok = whole || (tok0 + ((uint32_t)rb << (M - 7))) * (uint32_t)P::C < valid;
#pragma unroll
            for (int nb = 0; nb < P::NNB; ++nb) {
                f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int p = 0; p < NP; ++p) {
                    const f32x4 a = wf[(nb * NP + p) * 64 + lane];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            a[e], v[(4 * p + e) | (rb << RB_SHIFT)], acc, 0, 0, 0);
                }
                // channels 16 nb + 4 q + [0, 4)
                const u32x4 d = __builtin_bit_cast(u32x4, acc);
                if (ok)
                    __builtin_amdgcn_raw_buffer_store_b128(d, r, row + 16u * q,
                                                           rb * rb_bytes + 64u * nb, kYPolicy);
            }
        }
    }
}

// Stores Z' itself (float32, row-major like y) from the epilogue layout of a
// 2^M tile, through LDS into layout M-5, whose registers each cover 2^(M-5)
// consecutive elements (the epilogue layout's own stores would write 16 bytes
// to each of 64 lines per instruction).  Waits for earlier readers of the
// LDS first; the caller synchronises before the LDS is written again.
template <int M, int CB>
__device__ __forceinline__ void store_epilogue_f32(float *lds, const float (&v)[V], float *tile,
                                                   uint32_t valid, uint32_t tau)
{
    using E = Epi<M, CB>;
    const uint32_t pe = pad(E::base(tau));
    __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pe + pad(reg_offset<E>((uint32_t)k))] = v[k];
    __syncthreads();
    float u[V];
    const uint32_t ps = pad(layout_base<M - 5>(tau));
#pragma unroll
    for (int k = 0; k < V; ++k)
        u[k] = lds[ps + pad((uint32_t)k << (M - 5))];
    store_tile<M - 5, M, float>(u, tile, valid, tau);
}

// ---------------------------------------------------------------- LDS plan
// The tile's exchanges use pad(2^M) floats.  The prologue's weights share
// that space (they are dead before the first exchange).  The epilogue's
// weights either get their own region, loaded at kernel start, or share it
// too, prefetched into registers at start and written to LDS after the last
// exchange; sharing is chosen when a private region would cost occupancy and
// the prefetch takes at most 8 16-byte registers per thread.
template <int M, typename T, int CB>
struct Lds {
    static constexpr uint32_t NT = 1u << (M - VB);
    static constexpr uint32_t TILE = pad(1u << M) * 4u;
    static constexpr uint32_t W = Proj<T, CB>::WBYTES;
    static constexpr uint32_t CHUNKS = W / 16u;
    static constexpr bool PREFETCH_OK = CHUNKS % NT == 0 && CHUNKS / NT <= 8;
    static constexpr bool SEPARATE = TILE + W <= 80u * 1024u || !PREFETCH_OK;
    static constexpr uint32_t PER = PREFETCH_OK ? CHUNKS / NT : 1;
    static constexpr uint32_t REGION0 = TILE > W ? TILE : W;   // tile, or weights first
    static constexpr uint32_t fwd_bytes() { return REGION0; }
    static constexpr uint32_t inv_bytes() { return SEPARATE ? TILE + W : REGION0; }
    static constexpr uint32_t fused_bytes() { return SEPARATE ? REGION0 + W : REGION0; }
};

template <uint32_t CHUNKS, uint32_t NT>
__device__ __forceinline__ void stage_weights(void *lds, const void *w, uint32_t tau)
{
    u32x4 *d = static_cast<u32x4 *>(lds);
    const u32x4 *s = static_cast<const u32x4 *>(w);
    // Chunks tau, tau + NT, ... below CHUNKS, over a compile-time trip count so
    // the copy unrolls (a tau-dependent count left it a loop; the float32
    // block on 32 slices of 2^18 took 64 us per call then, 58 now, and on 2
    // slices of 2^21 58 then, 51 now).
#pragma unroll
    for (uint32_t i = 0; i < (CHUNKS + NT - 1) / NT; ++i) {
        const uint32_t c = tau + i * NT;
        if (CHUNKS % NT == 0 || c < CHUNKS)
            d[c] = s[c];
    }
}

// The same copy without a trip through registers (global_load_lds_dwordx4):
// piece c = tau + i NT lands at byte 16 c, so each wave's 64 pieces of a step
// are contiguous from a wave-uniform base, the instruction's LDS pattern.
// The caller waits (vmcnt) and synchronises before reading.
template <uint32_t CHUNKS, uint32_t NT>
__device__ __forceinline__ void stage_weights_dma(void *lds, const void *w, uint32_t tau)
{
    static_assert(CHUNKS % NT == 0 && NT % 64 == 0, "whole waves");
    const uint32_t wave = tau >> 6;
#pragma unroll
    for (uint32_t i = 0; i < CHUNKS / NT; ++i)
        __builtin_amdgcn_global_load_lds(
            static_cast<const char *>(w) + 16u * (tau + i * NT),
            static_cast<char *>(lds) + 16u * (wave * 64u + i * NT), 16, 0, 0);
}

// ---------------------------------------------------------------- kernels
// FUSED: one workgroup per slice (M = K).
template <int K, typename T, class Gain, int CB>
__global__ void __launch_bounds__(1 << (K - VB))
module_fused_kernel(const T *__restrict__ x, const T *__restrict__ w_in,
                    const T *__restrict__ w_out, T *__restrict__ y, Gain gain, uint32_t nvalid)
{
    using L = Lds<K, T, CB>;
    __shared__ __attribute__((aligned(16))) float lds[L::fused_bytes() / 4];
    unsigned char *const region1 = reinterpret_cast<unsigned char *>(lds) + L::REGION0;
    const uint32_t tau = threadIdx.x;
    const size_t base = (size_t)blockIdx.x * nvalid;
    XFrag<T, CB> f;
    load_x_frags<T, CB>(f, x + base, nvalid, nvalid >= (1u << K), tau);
    stage_weights<L::CHUNKS, L::NT>(lds, w_in, tau);
    u32x4 wreg[L::PER];
    if constexpr (L::SEPARATE) {
        stage_weights<L::CHUNKS, L::NT>(region1, w_out, tau);
    } else {
#pragma unroll
        for (uint32_t i = 0; i < L::PER; ++i)
            wreg[i] = static_cast<const u32x4 *>(static_cast<const void *>(w_out))[tau + i * L::NT];
    }
    float v[V], gv[V];
    gain.template load<K - 5, ContigMap>(gv, 0, tau);
    __syncthreads();
    project_in<T, CB>(v, f, lds, tau);
    forward_from_prologue<K>(lds, v, tau);
    apply_gain<K>(v, gv);
    inverse_to_epilogue<K, CB, true>(lds, v, tau);
    const void *wl = region1;
    if constexpr (!L::SEPARATE) {
        __syncthreads();   // every thread has read its epilogue-layout values
#pragma unroll
        for (uint32_t i = 0; i < L::PER; ++i)
            reinterpret_cast<u32x4 *>(lds)[tau + i * L::NT] = wreg[i];
        wl = lds;
    }
    __syncthreads();
    project_out<T, CB, K>(v, wl, y + base, nvalid, tau);
}

// THREE_PASS first pass: prologue, forward over the A low bits, workspace.
template <int A, int HB, int R, typename T, int CB>
__device__ __forceinline__ void module_outer_fwd_tile(float *lds, const T *__restrict__ x,
                                                      const T *__restrict__ w_in,
                                                      float *__restrict__ ws, uint32_t nvalid,
                                                      uint32_t blk)
{
    using L = Lds<A, T, CB>;
    using Run = RunMap<HB, R>;
    const uint32_t tau = threadIdx.x;
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const uint32_t valid = tile_valid<A>(nvalid, hi);
    XFrag<T, CB> f;
    load_x_frags<T, CB>(f, x + b * nvalid + ((size_t)hi << A), valid, valid >= (1u << A), tau);
    stage_weights<L::CHUNKS, L::NT>(lds, w_in, tau);
    __syncthreads();
    float v[V];
    project_in<T, CB>(v, f, lds, tau);
    forward_from_prologue<A>(lds, v, tau);
    store_layout<A - 5, Run, float>(
        v, buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>()), tau);
}

template <int A, int HB, int R, typename T, int CB>
__global__ void __launch_bounds__(1 << (A - VB))
module_outer_fwd_kernel(const T *__restrict__ x, const T *__restrict__ w_in,
                        float *__restrict__ ws, uint32_t nvalid)
{
    __shared__ __attribute__((aligned(16))) float lds[Lds<A, T, CB>::fwd_bytes() / 4];
    module_outer_fwd_tile<A, HB, R, T, CB>(lds, x, w_in, ws, nvalid,
                                           outer_block<R>(blockIdx.x, gridDim.x));
}

// Two operands in one launch (the block's backward: Z = X W_in and
// dZ' = dY W_out^T): the first half of the grid takes (x, wa) into wsx, the
// second (dy, wb) into wsd, each half numbered as a grid of its own.
template <int A, int HB, int R, typename T, int CB>
__global__ void __launch_bounds__(1 << (A - VB))
module_outer_fwd2_kernel(const T *__restrict__ x, const T *__restrict__ wa,
                         const T *__restrict__ dy, const T *__restrict__ wb,
                         float *__restrict__ wsx, float *__restrict__ wsd, uint32_t nvalid)
{
    __shared__ __attribute__((aligned(16))) float lds[Lds<A, T, CB>::fwd_bytes() / 4];
    const uint32_t half = gridDim.x >> 1;
    const bool second = blockIdx.x >= half;
    const uint32_t blk = outer_block<R>(blockIdx.x - (second ? half : 0u), half);
    module_outer_fwd_tile<A, HB, R, T, CB>(lds, second ? dy : x, second ? wb : wa,
                                           second ? wsd : wsx, nvalid, blk);
}

// THREE_PASS last pass: inverse over the A low bits, epilogue, y.  ZOUT: also
// store the inverse-transformed tile itself (float32) to z.
template <int A, int HB, int R, typename T, int CB, bool ZOUT = false>
__global__ void __launch_bounds__(1 << (A - VB))
module_outer_inv_kernel(const float *__restrict__ ws, const T *__restrict__ w_out,
                        T *__restrict__ y, float *__restrict__ z, uint32_t nvalid)
{
    using L = Lds<A, T, CB>;
    using Run = RunMap<HB, R>;
    __shared__ __attribute__((aligned(16))) float lds[L::inv_bytes() / 4];
    unsigned char *const wregion = reinterpret_cast<unsigned char *>(lds) + L::TILE;
    const uint32_t tau = threadIdx.x;
    const uint32_t blk = outer_block<R>(blockIdx.x, gridDim.x);
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const uint32_t valid = tile_valid<A>(nvalid, hi);
    if (valid == 0)
        return;   // wholly padding: nothing to store (uniform per workgroup)
    u32x4 wreg[L::PER];
    if constexpr (L::SEPARATE) {
        stage_weights<L::CHUNKS, L::NT>(wregion, w_out, tau);
    } else {
#pragma unroll
        for (uint32_t i = 0; i < L::PER; ++i)
            wreg[i] = static_cast<const u32x4 *>(static_cast<const void *>(w_out))[tau + i * L::NT];
    }
    float v[V];
    load_layout<A - 5, Run, float>(
        v, buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>()), tau);
    inverse_to_epilogue<A, CB, false>(lds, v, tau);
    if constexpr (ZOUT)
        store_epilogue_f32<A, CB>(lds, v, z + b * nvalid + ((size_t)hi << A), valid, tau);
    const void *wl = wregion;
    if constexpr (!L::SEPARATE) {
        __syncthreads();
#pragma unroll
        for (uint32_t i = 0; i < L::PER; ++i)
            reinterpret_cast<u32x4 *>(lds)[tau + i * L::NT] = wreg[i];
        wl = lds;
    }
    __syncthreads();
    project_out<T, CB, A>(v, wl, y + b * nvalid + ((size_t)hi << A), valid, tau);
}

// ---------------------------------------------------------------- C = 256 (bf16)
// Outer tiles of 2^16 elements = 256 tokens x 256 channels (t = token * 256 +
// channel), 1024 threads of two 2^15 register sets (pair_split).  Wave w owns
// 16 tokens, one 16-row MFMA block, against all 256 channels: 16 column
// blocks x 4 results = 64 values per lane, exactly the two sets.
//
// Forward: MFMA row m = 4q + r of wave w is token
//     (r & 1) | q << 1 | w << 3 | (r >> 1) << 7,
// so set s = t bit 15 (token bit 7) and within a set register nb | (r & 1) << 4
// holds t bits 4-8 (channel block nb, token bit 0) while lanes 0-3 (column j)
// hold channel bits 0-3, lanes 4-5 (q) t bits 9-10 and waves t bits 11-14:
// layout 4 of the set's 2^15 elements, as for C <= 128.  Bit 15 is a register
// butterfly between the sets.
//
// Inverse: set s = t bit 5 (channel bit 5).  Dropping that bit (t') leaves a
// 2^15 set laid out like a C = 128 tile, so the C = 128 inverse schedule ends
// in the epilogue layout Epi<15, 7>: lane (j, q) of wave w holds channels
// 64 q + 32 s + [0, 32) of token j | w << 4, the B operand of
// Y^T = W_out^T Z'^T.
//
// Both products use v_mfma_f32_16x16x32_bf16 (lane 16 g + i supplies k = 8 g
// + [0, 8) of row i of A / column i of B), half the instructions of the
// 16x16x16 form: step kk of the prologue is channels 32 kk + 8 g + [0, 8) (one
// 16-byte load of x), of the epilogue channels 64 g + 8 kk + [0, 8).
constexpr int kPairCB = kPairModuleCbits;
constexpr uint32_t kPairC = 1u << kPairCB;
constexpr uint32_t kPairThreads = 1u << (15 - VB);
constexpr uint32_t kPairKs = kPairC / 32u;                      // k steps
constexpr uint32_t kPairWChunks = kPairC * kPairC * 2u / 16u;   // 16-byte pieces of W

static_assert(kPairC * kPairC * 2u <= pad(1u << 15) * 4u, "W fits the tile's LDS");
static_assert(kPairWChunks % kPairThreads == 0, "whole pieces of W per thread");

// Set-local index t' (t bit 5 dropped) -> workspace offset.
template <class Map>
struct DropBit5 {
    __host__ __device__ static constexpr uint32_t at(uint32_t tp)
    {
        return Map::at((tp & 31u) | ((tp >> 5) << 6));
    }
};

// X fragments of the wave's 16 tokens: k step kk holds channels
// 32 kk + 8 q + [0, 8).
__device__ __forceinline__ void load_x_pair(bf16x8 (&a)[kPairKs], const __bf16 *tile,
                                            uint32_t valid, uint32_t tau)
{
    const uint32_t lane = tau & 63u, w = tau >> 6;
    const uint32_t i = lane & 15u, q = lane >> 4;
    const uint32_t tok = (i & 1u) | (((i >> 2) & 3u) << 1) | (w << 3) | (((i >> 1) & 1u) << 7);
    const bool ok = tok * kPairC < valid;
    const __amdgpu_buffer_rsrc_t r = buffer(tile, valid * 2u);
    const uint32_t voff = tok * kPairC * 2u + 16u * q;
#pragma unroll
    for (uint32_t kk = 0; kk < kPairKs; ++kk) {
        u32x4 d = {0u, 0u, 0u, 0u};
        if (ok)
            d = __builtin_amdgcn_raw_buffer_load_b128(r, voff, 64u * kk, kStreaming);
        a[kk] = __builtin_bit_cast(bf16x8, d);
    }
}

// Z = X W_in into the two sets (packed W_in in LDS).
__device__ __forceinline__ void project_in_pair(float (&v0)[V], float (&v1)[V],
                                                const bf16x8 (&a)[kPairKs], const void *wl,
                                                uint32_t tau)
{
    const bf16x8 *wb = static_cast<const bf16x8 *>(wl);
    const uint32_t lane = tau & 63u;
#pragma unroll
    for (int nb = 0; nb < 16; ++nb) {
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (uint32_t kk = 0; kk < kPairKs; ++kk)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[kk], wb[(nb * kPairKs + kk) * 64u + lane],
                                                          acc, 0, 0, 0);
        v0[nb] = acc[0];
        v0[nb | 16] = acc[1];
        v1[nb] = acc[2];
        v1[nb | 16] = acc[3];
    }
}

// The two-term split Z' = hi + lo of the two sets' epilogue-layout registers,
// as B operands: step kk element e is channel 64 q + 8 kk + e, i.e. set
// kk / 4, register 8 (kk % 4) + e.
__device__ __forceinline__ void split_pair(const float (&v0)[V], const float (&v1)[V],
                                           bf16x8 (&hi)[kPairKs], bf16x8 (&lo)[kPairKs])
{
#pragma unroll
    for (uint32_t kk = 0; kk < kPairKs; ++kk) {
        u32x4 h2, l2;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float z0 = kk < 4 ? v0[8 * kk + 2 * e] : v1[8 * (kk - 4) + 2 * e];
            const float z1 = kk < 4 ? v0[8 * kk + 2 * e + 1] : v1[8 * (kk - 4) + 2 * e + 1];
            const float h0 = (float)(__bf16)z0, h1 = (float)(__bf16)z1;
            h2[e] = pack2_bf16(z0, z1);
            l2[e] = pack2_bf16(z0 - h0, z1 - h1);
        }
        hi[kk] = __builtin_bit_cast(bf16x8, h2);
        lo[kk] = __builtin_bit_cast(bf16x8, l2);
    }
}

// Y = Z' W_out for the wave's 16 tokens (packed W_out in LDS); rows past
// `valid` are not stored.
__device__ __forceinline__ void project_out_pair(const bf16x8 (&hi)[kPairKs],
                                                 const bf16x8 (&lo)[kPairKs], const void *wl,
                                                 __bf16 *tile, uint32_t valid, uint32_t tau)
{
    const bf16x8 *wb = static_cast<const bf16x8 *>(wl);
    const uint32_t lane = tau & 63u, w = tau >> 6;
    const uint32_t j = lane & 15u, q = lane >> 4;
    const uint32_t tok = j | (w << 4);
    const bool ok = tok * kPairC < valid;
    const __amdgpu_buffer_rsrc_t r = buffer(tile, valid * 2u);
    const uint32_t voff = tok * kPairC * 2u + 16u * q;
    // blocks 2n, 2n+1: channels 32 n + 8 q + [0, 8), one 16-byte store
#pragma unroll
    for (uint32_t n = 0; n < 8; ++n) {
        f32x4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (uint32_t kk = 0; kk < kPairKs; ++kk) {
            const bf16x8 a0 = wb[((2 * n) * kPairKs + kk) * 64u + lane];
            const bf16x8 a1 = wb[((2 * n + 1) * kPairKs + kk) * 64u + lane];
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, hi[kk], acc0, 0, 0, 0);
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, lo[kk], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, hi[kk], acc1, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, lo[kk], acc1, 0, 0, 0);
        }
        const u32x4 d = {pack2_bf16(acc0[0], acc0[1]), pack2_bf16(acc0[2], acc0[3]),
                         pack2_bf16(acc1[0], acc1[1]), pack2_bf16(acc1[2], acc1[3])};
        if (ok)
            __builtin_amdgcn_raw_buffer_store_b128(d, r, voff, 64u * n, kYPolicy);
    }
}

// THREE_PASS first pass, C = 256: prologue, forward over the 16 low bits.
template <int HB, int R>
__device__ __forceinline__ void module_outer_fwd_pair_tile(float *lds, const __bf16 *__restrict__ x,
                                                           const __bf16 *__restrict__ w_in,
                                                           float *__restrict__ ws,
                                                           uint32_t nvalid, uint32_t blk)
{
    constexpr int A = 16, M = 15;
    using Run = RunMap<HB, R>;
    const uint32_t tau = threadIdx.x;
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const uint32_t valid = tile_valid<A>(nvalid, hi);
    bf16x8 a[kPairKs];
    load_x_pair(a, x + b * nvalid + ((size_t)hi << A), valid, tau);
    stage_weights_dma<kPairWChunks, kPairThreads>(lds, w_in, tau);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    float v0[V], v1[V];
    project_in_pair(v0, v1, a, lds, tau);
    cross_butterflies(v0, v1);   // bit 15
    const __amdgpu_buffer_rsrc_t r =
        buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>());
    forward_from_prologue<M>(lds, v0, tau);
    store_layout<M - 5, Run, float>(v0, r, tau);
    forward_from_prologue<M>(lds, v1, tau);
    store_layout<M - 5, Run, float>(v1, r, tau, Run::at(1u << M) * 4u);
}

template <int HB, int R>
__global__ void __launch_bounds__(kPairThreads)
module_outer_fwd_pair_kernel(const __bf16 *__restrict__ x, const __bf16 *__restrict__ w_in,
                             float *__restrict__ ws, uint32_t nvalid)
{
    __shared__ __attribute__((aligned(16))) float lds[pad(1u << 15)];
    module_outer_fwd_pair_tile<HB, R>(lds, x, w_in, ws, nvalid,
                                      outer_block<R>(blockIdx.x, gridDim.x));
}

// Two operands in one launch (the block's backward), as module_outer_fwd2_kernel.
template <int HB, int R>
__global__ void __launch_bounds__(kPairThreads)
module_outer_fwd2_pair_kernel(const __bf16 *__restrict__ x, const __bf16 *__restrict__ wa,
                              const __bf16 *__restrict__ dy, const __bf16 *__restrict__ wb,
                              float *__restrict__ wsx, float *__restrict__ wsd, uint32_t nvalid)
{
    __shared__ __attribute__((aligned(16))) float lds[pad(1u << 15)];
    const uint32_t half = gridDim.x >> 1;
    const bool second = blockIdx.x >= half;
    const uint32_t blk = outer_block<R>(blockIdx.x - (second ? half : 0u), half);
    module_outer_fwd_pair_tile<HB, R>(lds, second ? dy : x, second ? wb : wa, second ? wsd : wsx,
                                      nvalid, blk);
}

// Stores one set's inverse-transformed elements (float32, row-major like y)
// from the epilogue layout, through LDS into layout 10 of the set (t bit 5 =
// s dropped): each register then covers 2^10 set elements in runs of 32
// consecutive floats.  Waits for earlier readers of the LDS first.
__device__ __forceinline__ void store_pair_set_f32(float *lds, const float (&v)[V], float *tile,
                                                   uint32_t valid, uint32_t s, uint32_t tau)
{
    using E = Epi<15, 7>;
    using Map = DropBit5<ContigMap>;
    const uint32_t pe = pad(E::base(tau));
    __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pe + pad(reg_offset<E>((uint32_t)k))] = v[k];
    __syncthreads();
    const uint32_t tb = layout_base<10>(tau);
    const uint32_t ps = pad(tb);
    // set element t' < valid / 2 holds token t' / 128 < valid / 256: a real row
    const __amdgpu_buffer_rsrc_t r = buffer(tile, valid * 4u);
    const uint32_t voff = (Map::at(tb) + (s << 5)) * 4u;
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const float u = lds[ps + pad((uint32_t)k << 10)];
        if ((tb | ((uint32_t)k << 10)) < valid / 2u)
            Elt<float>::store<kStreaming>(u, r, voff, Map::at((uint32_t)k << 10) * 4u);
    }
}

// THREE_PASS last pass, C = 256: inverse over the 16 low bits, epilogue, y.
// ZOUT: also store the inverse-transformed tile itself (float32) to z.
template <int HB, int R, bool ZOUT = false>
__global__ void __launch_bounds__(kPairThreads)
module_outer_inv_pair_kernel(const float *__restrict__ ws, const __bf16 *__restrict__ w_out,
                             __bf16 *__restrict__ y, float *__restrict__ z, uint32_t nvalid)
{
    constexpr int A = 16, M = 15;
    using Run = RunMap<HB, R>;
    using SetMap = DropBit5<Run>;
    __shared__ __attribute__((aligned(16))) float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t blk = outer_block<R>(blockIdx.x, gridDim.x);
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const uint32_t valid = tile_valid<A>(nvalid, hi);
    if (valid == 0)
        return;   // wholly padding: nothing to store (uniform per workgroup)
    const __amdgpu_buffer_rsrc_t r =
        buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>());
    float v0[V], v1[V];
    load_layout<M - 5, SetMap, float>(v0, r, tau);
    load_layout<M - 5, SetMap, float>(v1, r, tau, Run::at(1u << 5) * 4u);
    cross_butterflies(v0, v1);   // t bit 5 (the bit groups commute)
    inverse_to_epilogue<M, 7, false>(lds, v0, tau);
    inverse_to_epilogue<M, 7, true>(lds, v1, tau);
    if constexpr (ZOUT) {
        float *zt = z + b * nvalid + ((size_t)hi << A);
        store_pair_set_f32(lds, v0, zt, valid, 0u, tau);
        store_pair_set_f32(lds, v1, zt, valid, 1u, tau);
    }
    __syncthreads();             // every thread has read its epilogue-layout values
    stage_weights_dma<kPairWChunks, kPairThreads>(lds, w_out, tau);
    bf16x8 zh[kPairKs], zl[kPairKs];
    split_pair(v0, v1, zh, zl);  // while W_out arrives
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    project_out_pair(zh, zl, lds, y + b * nvalid + ((size_t)hi << A), valid, tau);
}

// The same pass as a grid of one resident workgroup per CU (the kernel's LDS
// holds W_out or the exchange, 128 KiB, so no second workgroup fits) taking
// tiles t, t + grid, ...: the first NPF of the 32 registers of the next
// tile's first set are read from the workspace while this tile's projection
// runs on the matrix cores, which otherwise leave the CU's memory path idle
// (more spill beside the projection's operands).  The read is issued after W_out
// has landed in LDS (the wait for it would also wait for the read) and kept
// ahead of the MFMAs by a scheduling barrier.
template <int HB, int R>
__global__ void __launch_bounds__(kPairThreads)
module_outer_inv_pair_pf_kernel(const float *__restrict__ ws, const __bf16 *__restrict__ w_out,
                                __bf16 *__restrict__ y, uint32_t nvalid, uint32_t ntiles)
{
    constexpr int A = 16, M = 15, NPF = 8;
    using Run = RunMap<HB, R>;
    using SetMap = DropBit5<Run>;
    __shared__ __attribute__((aligned(16))) float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t voff = SetMap::at(layout_base<M - 5>(tau)) * 4u;
    auto tile_ws = [&](uint32_t blk) {
        return buffer(ws + ((size_t)(blk >> HB) << (A + HB)) +
                          ((size_t)(blk & ((1u << HB) - 1u)) << R),
                      extent_bytes<Run, A, float>());
    };
    // register k of set s (as load_layout<M - 5, SetMap> with the set's offset)
    auto read = [&](__amdgpu_buffer_rsrc_t r, int k, uint32_t s) {
        return Elt<float>::load<kTemporal>(
            r, voff, s * Run::at(1u << 5) * 4u + SetMap::at((uint32_t)k << (M - 5)) * 4u);
    };
    float nx[NPF];
    uint32_t t = blockIdx.x;
    if (t < ntiles) {
        const __amdgpu_buffer_rsrc_t r = tile_ws(outer_block<R>(t, ntiles));
#pragma unroll
        for (int k = 0; k < NPF; ++k)
            nx[k] = read(r, k, 0u);
    }
    for (; t < ntiles; t += gridDim.x) {   // uniform per workgroup
        const uint32_t blk = outer_block<R>(t, ntiles);
        const size_t b = blk >> HB;
        const uint32_t hi = blk & ((1u << HB) - 1u);
        const uint32_t valid = tile_valid<A>(nvalid, hi);
        const bool more = t + gridDim.x < ntiles;
        const __amdgpu_buffer_rsrc_t rn =
            tile_ws(more ? outer_block<R>(t + gridDim.x, ntiles) : blk);
        if (valid == 0) {   // wholly padding: nothing to store
            if (more) {
#pragma unroll
                for (int k = 0; k < NPF; ++k)
                    nx[k] = read(rn, k, 0u);
            }
            continue;
        }
        float v0[V], v1[V];
        {
            const __amdgpu_buffer_rsrc_t r = tile_ws(blk);
#pragma unroll
            for (int k = 0; k < V; ++k)
                v0[k] = k < NPF ? nx[k] : read(r, k, 0u);
#pragma unroll
            for (int k = 0; k < V; ++k)
                v1[k] = read(r, k, 1u);
        }
        cross_butterflies(v0, v1);   // t bit 5 (the bit groups commute)
        inverse_to_epilogue<M, 7, true>(lds, v0, tau);   // the last tile's W_out readers first
        inverse_to_epilogue<M, 7, true>(lds, v1, tau);
        __syncthreads();             // every thread has read its epilogue-layout values
        stage_weights_dma<kPairWChunks, kPairThreads>(lds, w_out, tau);
        bf16x8 zh[kPairKs], zl[kPairKs];
        split_pair(v0, v1, zh, zl);  // while W_out arrives
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (more) {
#pragma unroll
            for (int k = 0; k < NPF; ++k)
                nx[k] = read(rn, k, 0u);
        }
        __builtin_amdgcn_sched_barrier(0);
        project_out_pair(zh, zl, lds, y + b * nvalid + ((size_t)hi << A), valid, tau);
    }
}

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(__bf16 v) { return (float)v; }

// SMALL: 2^K <= 2^10, one 256-thread workgroup per slice, everything in LDS,
// projections on the VALU (any C).
template <typename T, class Gain>
__global__ void __launch_bounds__(256)
module_small_kernel(const T *__restrict__ x, const T *__restrict__ w_in,
                    const T *__restrict__ w_out, T *__restrict__ y, Gain gain, int K, int cb,
                    uint32_t nvalid)
{
    __shared__ float xs[1 << kMaxSmall];
    __shared__ float s[1 << kMaxSmall];
    const int L = 1 << K;
    const uint32_t C = 1u << cb;
    const size_t base = (size_t)blockIdx.x * nvalid;
    for (int i = threadIdx.x; i < L; i += blockDim.x)
        xs[i] = (uint32_t)i < nvalid ? to_f(x[base + i]) : 0.0f;
    __syncthreads();
    for (int i = threadIdx.x; i < L; i += blockDim.x) {
        const uint32_t row = (uint32_t)i >> cb, c = (uint32_t)i & (C - 1u);
        float acc = 0.0f;
        for (uint32_t k = 0; k < C; ++k)
            acc = fmaf(xs[row * C + k], to_f(w_in[k * C + c]), acc);
        s[i] = acc;
    }
    const float scale = 1.0f / (float)L;
    for (int pass = 0; pass < 2; ++pass) {
        for (int h = 1; h < L; h <<= 1) {
            __syncthreads();
            for (int p = threadIdx.x; p < L / 2; p += blockDim.x) {
                const int i = ((p / h) * 2 * h) + (p % h);
                const float a = s[i], c = s[i + h];
                s[i] = a + c;
                s[i + h] = a - c;
            }
        }
        __syncthreads();
        if (pass == 0)
            for (int i = threadIdx.x; i < L; i += blockDim.x)
                s[i] *= gain.at((uint32_t)i) * scale;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < (int)nvalid; i += blockDim.x) {
        const uint32_t row = (uint32_t)i >> cb, c = (uint32_t)i & (C - 1u);
        float acc = 0.0f;
        for (uint32_t k = 0; k < C; ++k)
            acc = fmaf(s[row * C + k], to_f(w_out[k * C + c]), acc);
        y[base + i] = (T)acc;
    }
}

// UNFUSED projection: out[row][c] = sum_k in[row][k] w[k][c], one thread per
// output, for the channel counts the MFMA layouts do not cover.
template <typename Tin, typename Tout, typename Tw, bool TRANS = false>
__global__ void __launch_bounds__(256)
project_rows_kernel(const Tin *__restrict__ in, const Tw *__restrict__ w, Tout *__restrict__ out,
                    uint64_t total, int cb)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256u + threadIdx.x;
    if (i >= total) return;
    const uint32_t C = 1u << cb;
    const uint32_t c = (uint32_t)(i & (C - 1u));
    const Tin *row = in + (i - c);
    float acc = 0.0f;
    for (uint32_t k = 0; k < C; ++k)   // TRANS: out = in W^T
        acc = fmaf(to_f(row[k]), to_f(TRANS ? w[(size_t)c * C + k] : w[(size_t)k * C + c]), acc);
    out[i] = (Tout)acc;
}

// Projection on the matrix cores, out[row][c] = sum_k in[row][k] W[k][c], for
// C >= 32: the UNFUSED forward (C >= 256; the fused layouts cover 16..128)
// and the block's backward.  W is packed in the prologue's operand order, where
// the NCOL columns of a slice are contiguous.
// Workgroup (g, slice) stages its slice into LDS once and loops over blocks of
// 64 rows, 16 per wave.  Operands as in the prologue: bf16 rows against bf16
// weights; float rows against bf16 weights split as hi + lo; float against
// float on the fp32 instruction.
template <typename Tw, int CB>
struct ProjCols {
    static constexpr int C = 1 << CB;
    static constexpr int raw = 65536 / (C * (int)sizeof(Tw));
    static constexpr int cap = C < 128 ? C : 128;   // columns of one slice
    static constexpr int NCOL = raw > cap ? cap : (raw < 16 ? 16 : raw);
    static constexpr uint32_t WSLICE = (uint32_t)C * NCOL * sizeof(Tw);
    static constexpr bool OK = WSLICE <= 128u * 1024u && C >= 32;
};

__device__ __forceinline__ void split_bf16(const f32x4 &z, bf16x4 &hi, bf16x4 &lo)
{
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const __bf16 h = (__bf16)z[e];
        hi[e] = __builtin_bit_cast(short, h);
        lo[e] = __builtin_bit_cast(short, (__bf16)(z[e] - (float)h));
    }
}

// Operand pieces of the projection kernel: one 16-byte load per lane per
// piece.  bf16 rows: piece p holds channels 32p + 8q + [0, 8), the k values of
// steps 2p and 2p+1.  Float rows: piece u holds 4 channels, 32(u/2) + 8q +
// 4(u%2) + [0, 4) against bf16 weights (step u) or 16u + 4q + [0, 4) against
// float weights (steps 4u .. 4u+3).  A chunk is CH = min(C, 256) channels of
// a row (offsets below are within the chunk).
template <typename Tin, typename Tw, int C>
struct ProjMode {
    static constexpr bool BFW = sizeof(Tw) == 2;
    static constexpr bool BFIN = sizeof(Tin) == 2;
    static constexpr int CH = C < 256 ? C : 256;
    static constexpr int NPC = BFIN ? CH / 32 : CH / 16;   // pieces per chunk
    __device__ static uint32_t channel(uint32_t piece, uint32_t q)
    {
        if constexpr (BFIN) return 32u * piece + 8u * q;
        else if constexpr (BFW) return 32u * (piece >> 1) + 8u * q + 4u * (piece & 1u);
        else return 16u * piece + 4u * q;
    }
};

template <typename Tin, typename Tout, typename Tw, int CB>
__global__ void __launch_bounds__(256)
project_mfma_kernel(const Tin *__restrict__ in, const Tw *__restrict__ wpk, Tout *__restrict__ out,
                    uint32_t rows)
{
    using PC = ProjCols<Tw, CB>;
    using PM = ProjMode<Tin, Tw, (1 << CB)>;
    constexpr int C = PC::C;
    constexpr int NB = PC::NCOL / 16;
    constexpr int KS = PM::BFW ? C / 16 : C / 4;   // k steps of one column block
    constexpr int NCH = C / PM::CH;                // chunks per row
    constexpr int NPC = PM::NPC;
    static_assert(PC::OK, "weight slice must fit LDS");
    __shared__ __attribute__((aligned(16))) unsigned char lds[PC::WSLICE];
    const uint32_t tau = threadIdx.x, lane = tau & 63u, w = tau >> 6;
    const uint32_t i = lane & 15u, q = lane >> 4;
    const uint32_t slice = blockIdx.y;
    // the slice's column blocks are contiguous in the packed matrix
    stage_weights<PC::WSLICE / 16, 256>(lds, wpk + (size_t)slice * PC::NCOL * C, tau);
    __syncthreads();

    // step t: row block blockIdx.x + (t / NCH) * gridDim.x, chunk t % NCH
    const uint32_t nblk = (rows + 63u) / 64u;
    const uint32_t mine = blockIdx.x < nblk ? (nblk - 1u - blockIdx.x) / gridDim.x + 1u : 0u;
    const uint32_t T = mine * NCH;
    auto load = [&](u32x4 (&buf)[NPC], uint32_t t) {
        const uint32_t blk = blockIdx.x + (t / NCH) * gridDim.x;
        const uint32_t row = blk * 64u + w * 16u + i;
        const uint32_t c0 = (t % NCH) * (uint32_t)PM::CH;
        const Tin *src = in + (size_t)row * C + c0;
#pragma unroll
        for (int u = 0; u < NPC; ++u) {
            buf[u] = (u32x4){0u, 0u, 0u, 0u};
            if (row < rows)
                buf[u] = *reinterpret_cast<const u32x4 *>(src + PM::channel(u, q));
        }
    };
    f32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
        acc[nb] = (f32x4){0.0f, 0.0f, 0.0f, 0.0f};
    auto compute = [&](const u32x4 (&buf)[NPC], uint32_t t) {
        const uint32_t ch = t % NCH;
        if constexpr (PM::BFW && PM::BFIN) {
            const bf16x4 *wb = reinterpret_cast<const bf16x4 *>(lds);
#pragma unroll
            for (int u = 0; u < NPC; ++u) {
                const uint32_t kk = 2u * (ch * NPC + u);
                const bf16x4 a0 = __builtin_bit_cast(bf16x4, (u32x2){buf[u].x, buf[u].y});
                const bf16x4 a1 = __builtin_bit_cast(bf16x4, (u32x2){buf[u].z, buf[u].w});
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
                        a0, wb[(nb * KS + kk) * 64 + lane], acc[nb], 0, 0, 0);
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
                        a1, wb[(nb * KS + kk + 1) * 64 + lane], acc[nb], 0, 0, 0);
                }
                // keep the weight reads of later pieces below this piece's MFMAs
                // (hoisting them all costs registers and occupancy)
                __builtin_amdgcn_sched_barrier(0);
            }
        } else if constexpr (PM::BFW) {
            const bf16x4 *wb = reinterpret_cast<const bf16x4 *>(lds);
#pragma unroll
            for (int u = 0; u < NPC; ++u) {
                const uint32_t kk = ch * NPC + u;
                bf16x4 hi, lo;
                split_bf16(__builtin_bit_cast(f32x4, buf[u]), hi, lo);
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const bf16x4 b = wb[(nb * KS + kk) * 64 + lane];
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(hi, b, acc[nb], 0, 0, 0);
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(lo, b, acc[nb], 0, 0, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        } else {
            const f32x4 *wf = reinterpret_cast<const f32x4 *>(lds);
#pragma unroll
            for (int u = 0; u < NPC; ++u) {
                const uint32_t p = ch * NPC + u;
                const f32x4 a = __builtin_bit_cast(f32x4, buf[u]);
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const f32x4 b = wf[(nb * (C / 16) + p) * 64 + lane];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], acc[nb], 0, 0,
                                                                       0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if (ch == NCH - 1) {
            // lane 16 q + j holds rows 4q + r of column 16 nb + j
            const uint32_t blk = blockIdx.x + (t / NCH) * gridDim.x;
            const uint32_t r0 = blk * 64u + w * 16u;
            const uint32_t col = slice * PC::NCOL + i;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t row = r0 + 4u * q + r;
                if (row < rows) {
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
                        out[(size_t)row * C + col + 16u * nb] = (Tout)acc[nb][r];
                }
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[nb] = (f32x4){0.0f, 0.0f, 0.0f, 0.0f};
        }
    };
    // two buffers: the next step's pieces load while this step computes
    u32x4 b0[NPC], b1[NPC];
    if (T > 0) load(b0, 0);
    for (uint32_t t = 0; t < T; t += 2) {
        if (t + 1 < T) load(b1, t + 1);
        compute(b0, t);
        if (t + 1 < T) {
            if (t + 2 < T) load(b0, t + 2);
            compute(b1, t + 1);
        }
    }
}

// ---------------------------------------------------------------- launchers
inline hipError_t record(hipEvent_t ev, hipStream_t st)
{
    return ev ? hipEventRecord(ev, st) : hipSuccess;
}

template <typename T>
hipError_t launch_pack(const ModuleArgs &m, bool out_as_in)
{
    const uint32_t n = 1u << (2 * m.cbits);
    hipLaunchKernelGGL((pack_weights_kernel<T>), dim3((n + 255u) / 256u), dim3(256), 0, m.stream,
                       static_cast<const T *>(m.w_in), static_cast<const T *>(m.w_out),
                       static_cast<T *>(m.wpack), static_cast<T *>(m.wpack) + n, m.cbits,
                       out_as_in ? 1 : 0);
    return hipGetLastError();
}

template <int K, typename T, class Gain, int CB>
hipError_t launch_module_fused(const ModuleArgs &m, Gain gain)
{
    const uint32_t n = 1u << (2 * CB);
    const T *pin = static_cast<const T *>(m.wpack);
    hipError_t e = record(m.events[0], m.stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((module_fused_kernel<K, T, Gain, CB>), dim3((uint32_t)m.B),
                       dim3(1u << (K - VB)), 0, m.stream, static_cast<const T *>(m.x), pin,
                       pin + n, static_cast<T *>(m.y), gain, m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(m.events[1], m.stream);
}

// Arguments of the mixer's middle pass inside the block's three-pass plan.
LaunchArgs middle_args(const ModuleArgs &m, bool pair_outer)
{
    LaunchArgs a{};
    a.gain_kind = m.gain_kind;
    a.gain = m.gain;
    a.gain_t = m.gain_t;
    a.gain_c = m.gain_c;
    a.cbits = m.cbits;
    a.ws = m.ws;
    a.B = m.B;
    a.K = m.K;
    a.plan = PLAN_THREE_PASS;
    a.stream = m.stream;
    a.pair_outer = pair_outer;
    return a;
}

template <int K, typename T, class Gain, int CB>
hipError_t launch_module_three_pass(const ModuleArgs &m, Gain gain)
{
    constexpr Split sp = module_split(K);
    constexpr int A = sp.A, HB = sp.HB, R = sp.R;
    const uint32_t n = 1u << (2 * CB);
    const T *pin = static_cast<const T *>(m.wpack);
    const hipStream_t st = m.stream;
    hipError_t e = record(m.events[0], st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((module_outer_fwd_kernel<A, HB, R, T, CB>), dim3((uint32_t)(m.B << HB)),
                       dim3(1u << (A - VB)), 0, st, static_cast<const T *>(m.x), pin, m.ws,
                       m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = record(m.events[1], st)) != hipSuccess) return e;
    if ((e = launch_middle(middle_args(m, false))) != hipSuccess) return e;
    if ((e = record(m.events[2], st)) != hipSuccess) return e;
    hipLaunchKernelGGL((module_outer_inv_kernel<A, HB, R, T, CB>), dim3((uint32_t)(m.B << HB)),
                       dim3(1u << (A - VB)), 0, st, m.ws, pin + n, static_cast<T *>(m.y),
                       nullptr, m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(m.events[3], st);
}

// C = 256 (bf16): the three passes on 2^16 outer tiles.
template <int K>
hipError_t launch_module_pair(const ModuleArgs &m)
{
    constexpr Split sp = pair_split(K);
    constexpr int HB = sp.HB, R = sp.R;
    static_assert(sp.A == 16 && HB >= 1, "pair split");
    const __bf16 *pin = static_cast<const __bf16 *>(m.wpack);
    const hipStream_t st = m.stream;
    const dim3 grid((uint32_t)(m.B << HB)), block(kPairThreads);
    hipError_t e = record(m.events[0], st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((module_outer_fwd_pair_kernel<HB, R>), grid, block, 0, st,
                       static_cast<const __bf16 *>(m.x), pin, m.ws, m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = record(m.events[1], st)) != hipSuccess) return e;
    if ((e = launch_middle(middle_args(m, true))) != hipSuccess) return e;
    if ((e = record(m.events[2], st)) != hipSuccess) return e;
    const uint32_t ntiles = (uint32_t)(m.B << HB);
    hipLaunchKernelGGL((module_outer_inv_pair_pf_kernel<HB, R>),
                       dim3(ntiles < 256u ? ntiles : 256u), block, 0, st, m.ws,
                       pin + kPairC * kPairC, static_cast<__bf16 *>(m.y), m.nvalid, ntiles);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(m.events[3], st);
}

hipError_t dispatch_pair(const ModuleArgs &m)
{
    switch (m.K) {
#define WHTMIX_MP_CASE(k) \
    case k: return launch_module_pair<k>(m);
        WHTMIX_MP_CASE(17) WHTMIX_MP_CASE(18) WHTMIX_MP_CASE(19) WHTMIX_MP_CASE(20)
        WHTMIX_MP_CASE(21) WHTMIX_MP_CASE(22) WHTMIX_MP_CASE(23) WHTMIX_MP_CASE(24)
        WHTMIX_MP_CASE(25) WHTMIX_MP_CASE(26) WHTMIX_MP_CASE(27) WHTMIX_MP_CASE(28)
        WHTMIX_MP_CASE(29) WHTMIX_MP_CASE(30)
#undef WHTMIX_MP_CASE
    default: return hipErrorInvalidValue;
    }
}

template <typename T, class Gain, int CB>
hipError_t dispatch_k(const ModuleArgs &m, Gain gain)
{
    if (m.plan == PLAN_FUSED) {
        switch (m.K) {
#define WHTMIX_MF_CASE(k) \
    case k: return launch_module_fused<k, T, Gain, CB>(m, gain);
            WHTMIX_MF_CASE(11) WHTMIX_MF_CASE(12) WHTMIX_MF_CASE(13) WHTMIX_MF_CASE(14)
            WHTMIX_MF_CASE(15)
#undef WHTMIX_MF_CASE
        default: return hipErrorInvalidValue;
        }
    }
    switch (m.K) {
#define WHTMIX_M3_CASE(k) \
    case k: return launch_module_three_pass<k, T, Gain, CB>(m, gain);
        WHTMIX_M3_CASE(12) WHTMIX_M3_CASE(13) WHTMIX_M3_CASE(14) WHTMIX_M3_CASE(15)
        WHTMIX_M3_CASE(16) WHTMIX_M3_CASE(17) WHTMIX_M3_CASE(18) WHTMIX_M3_CASE(19)
        WHTMIX_M3_CASE(20) WHTMIX_M3_CASE(21) WHTMIX_M3_CASE(22) WHTMIX_M3_CASE(23)
        WHTMIX_M3_CASE(24) WHTMIX_M3_CASE(25) WHTMIX_M3_CASE(26) WHTMIX_M3_CASE(27)
        WHTMIX_M3_CASE(28) WHTMIX_M3_CASE(29) WHTMIX_M3_CASE(30)
#undef WHTMIX_M3_CASE
    default: return hipErrorInvalidValue;
    }
}

template <typename T, class Gain>
hipError_t dispatch_fused_module(const ModuleArgs &m, Gain gain)
{
    hipError_t e;
    if (std::is_same<T, __bf16>::value && m.cbits >= 5) {
        const uint32_t n = 1u << (2 * m.cbits);
        const PackX32Jobs jobs{{static_cast<const __bf16 *>(m.w_in),
                                static_cast<const __bf16 *>(m.w_out), nullptr},
                               {static_cast<__bf16 *>(m.wpack),
                                static_cast<__bf16 *>(m.wpack) + n, nullptr},
                               {PACK_PROLOGUE, PACK_EPILOGUE, 0}};
        hipLaunchKernelGGL(pack_x32_kernel, dim3((n + 255u) / 256u), dim3(256), 0, m.stream, jobs,
                           m.cbits);
        e = hipGetLastError();
    } else {
        e = launch_pack<T>(m, false);
    }
    if (e != hipSuccess) return e;
    switch (m.cbits) {
    case 4: return dispatch_k<T, Gain, 4>(m, gain);
    case 5: return dispatch_k<T, Gain, 5>(m, gain);
    case 6: return dispatch_k<T, Gain, 6>(m, gain);
    case 7: return dispatch_k<T, Gain, 7>(m, gain);
    case kPairCB:
        if constexpr (std::is_same<T, __bf16>::value) return dispatch_pair(m);
        return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
    }
}

template <typename T, class Gain>
hipError_t launch_module_small(const ModuleArgs &m, Gain gain)
{
    hipError_t e = record(m.events[0], m.stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((module_small_kernel<T, Gain>), dim3((uint32_t)m.B), dim3(256), 0, m.stream,
                       static_cast<const T *>(m.x), static_cast<const T *>(m.w_in),
                       static_cast<const T *>(m.w_out), static_cast<T *>(m.y), gain, m.K, m.cbits,
                       m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(m.events[1], m.stream);
}

// UNFUSED: z = x W_in (fp32, in the workspace), the fp32 mixer in place on
// z, y = z W_out.  Projections on the matrix cores where a weight slice fits
// LDS (C >= 256 here), else one thread per output on the VALU.
template <typename T, int CB>
hipError_t project_pair_mfma(const ModuleArgs &m, LaunchArgs &mix)
{
    using PC = ProjCols<T, CB>;
    const uint32_t rows = (uint32_t)(((uint64_t)m.B * m.nvalid) >> CB);
    const uint32_t slices = PC::C / PC::NCOL;
    const uint32_t nblk = (rows + 63u) / 64u;
    uint32_t gx = 512u / slices;
    gx = gx < 1u ? 1u : (gx > nblk ? nblk : gx);
    const dim3 grid(gx, slices);
    const T *pin = static_cast<const T *>(m.wpack);
    const T *pout = pin + ((size_t)1 << (2 * CB));
    const hipStream_t st = m.stream;
    hipError_t e = launch_pack<T>(m, true);
    if (e != hipSuccess) return e;
    if ((e = record(m.events[0], st)) != hipSuccess) return e;
    hipLaunchKernelGGL((project_mfma_kernel<T, float, T, CB>), grid, dim3(256), 0, st,
                       static_cast<const T *>(m.x), pin, m.z, rows);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch(mix)) != hipSuccess) return e;
    hipLaunchKernelGGL((project_mfma_kernel<float, T, T, CB>), grid, dim3(256), 0, st, m.z, pout,
                       static_cast<T *>(m.y), rows);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(m.events[1], st);
}

template <typename T>
hipError_t launch_module_unfused(const ModuleArgs &m)
{
    const uint64_t total = (uint64_t)m.B * m.nvalid;
    const uint32_t blocks = (uint32_t)((total + 255u) / 256u);
    const hipStream_t st = m.stream;
    LaunchArgs a{};
    a.x = m.z;
    a.y = m.z;
    a.gain_kind = m.gain_kind;
    a.gain = m.gain;
    a.gain_t = m.gain_t;
    a.gain_c = m.gain_c;
    a.cbits = m.cbits;
    a.ws = m.ws;
    a.B = m.B;
    a.K = m.K;
    a.nvalid = m.nvalid;
    a.dtype = DTYPE_F32;
    a.plan = m.plan;
    a.stream = st;
    switch (m.cbits) {
#define WHTMIX_PM_CASE(cb) \
    case cb:               \
        if constexpr (ProjCols<T, cb>::OK && cb >= 8) return project_pair_mfma<T, cb>(m, a); \
        break;
        WHTMIX_PM_CASE(8) WHTMIX_PM_CASE(9) WHTMIX_PM_CASE(10) WHTMIX_PM_CASE(11)
        WHTMIX_PM_CASE(12)
#undef WHTMIX_PM_CASE
    default: break;
    }
    hipError_t e = record(m.events[0], st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((project_rows_kernel<T, float, T>), dim3(blocks), dim3(256), 0, st,
                       static_cast<const T *>(m.x), static_cast<const T *>(m.w_in), m.z, total,
                       m.cbits);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch(a)) != hipSuccess) return e;
    hipLaunchKernelGGL((project_rows_kernel<float, T, T>), dim3(blocks), dim3(256), 0, st, m.z,
                       static_cast<const T *>(m.w_out), static_cast<T *>(m.y), total, m.cbits);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(m.events[1], st);
}

template <typename T, class Gain>
hipError_t dispatch_module(const ModuleArgs &m, Gain gain)
{
    switch (module_path(m.plan, m.cbits, m.dtype, m.K)) {
    case MODULE_SMALL: return launch_module_small<T, Gain>(m, gain);
    case MODULE_FUSED_MFMA: return dispatch_fused_module<T, Gain>(m, gain);
    default: return launch_module_unfused<T>(m);
    }
}

template <typename T>
hipError_t dispatch_module_gain(const ModuleArgs &m)
{
    if (m.gain_kind == GAIN_LOG_SEPARABLE)
        return dispatch_module<T>(m, LogSeparableGain{m.gain_t, m.gain_c, (uint32_t)m.cbits});
    return dispatch_module<T>(m, FullGain{m.gain});
}


// ---------------------------------------------------------------- backward
// Gradients of the block (eqs. (1)-(4)) for an upstream gradient dY:
//   Z = X W_in and Z' = mixer(Z) are recomputed (float32);
//   dZ' = dY W_out^T;  dW_out = Z'^T dY;
//   dZ and the gain gradient: the mixer's own backward at (Z, dZ');
//   dX = dZ W_in^T;    dW_in = X^T dZ.
// Projections run on the matrix cores for C >= 32 (weights packed, transposed
// where the product needs W^T), on the VALU below.  Weight gradients use the
// fp32 16x16x4 MFMA, whose operand lanes (lane 16q + i: row q, column i of a
// 4 x 16 block) read row-major activations directly: each wave sums the
// products of one output tile over one chunk of rows, and the chunks' partial
// sums are added in a fixed order, so the result is reproducible.

// B-operand packing of W (TRANS: of W^T) in the prologue's order.
template <typename T>
__global__ void __launch_bounds__(256)
pack_b_kernel(const T *__restrict__ w, T *__restrict__ p, int cb, int trans)
{
    const uint32_t C = 1u << cb;
    const uint32_t idx = blockIdx.x * 256u + threadIdx.x;
    if (idx >= C * C) return;
    const uint32_t e = idx & 3u;
    const uint32_t lane = (idx >> 2) & 63u;
    const uint32_t j = lane & 15u, q = lane >> 4;
    const uint32_t rest = idx >> 8;
    uint32_t k, col;
    if constexpr (sizeof(T) == 2) {
        const uint32_t ks = C / 16u;
        k = k_in_bf16(C, rest % ks, q, e);
        col = 16u * (rest / ks) + j;
    } else {
        const uint32_t np = C / 16u;
        k = k_in_f32(4u * (rest % np) + e, q);
        col = 16u * (rest / np) + j;
    }
    p[idx] = trans ? w[col * C + k] : w[k * C + col];
}

// Partial dW = A^T B (A, B [rows][C]) of one chunk of rows on the matrix
// cores: one workgroup per (chunk, T x T block of dW), T = min(C, 128).
//
// Rows go through LDS in blocks of 64: 16-byte global loads, widened to
// float32 rows padded to LDW floats, the next block's loads issued before the
// current block's products.  Each wave owns a TQ x TQ quadrant of 16 x 16
// tiles (T = 16: wave 0 alone).  In one MFMA the lanes (i, q) hold, for
// k-slot e, the rows kb + q + 4e of column i: any assignment of rows to
// k-slots is a valid contraction order, and this one makes the four lane
// groups q read rows one apart, which LDW = T + 16 (48 for T = 16) puts on
// disjoint banks.
//
// Products (float32 accumulation):
//   float32 x float32: v_mfma_f32_16x16x4_f32, four rows per step;
//   bf16 x bf16:       v_mfma_f32_16x16x16_bf16, exact;
//   bf16 x float32:    the float is split into three bf16 terms (residual
//                      below 2^-27 |v|, finer than float32 itself) and each
//                      term goes through the bf16 instruction.
template <typename Ta, typename Tb, int T>
struct WgradShape {
    // rows per LDS block: 32 for float32 x float32 at T = 128, whose 64-row
    // prefetch would leave one workgroup per CU; 64 otherwise
    static constexpr int RB = sizeof(Ta) == 4 && sizeof(Tb) == 4 && T == 128 ? 32 : 64;
    static constexpr int LDW = T == 16 ? 48 : T + 16;      // padded LDS row (floats)
    static constexpr int TQ = T >= 32 ? T / 32 : 1;        // tiles per wave side
    static constexpr int VA = 16 / (int)sizeof(Ta);        // elements per 16-byte load
    static constexpr int VBL = 16 / (int)sizeof(Tb);
    static constexpr int NA = (RB * T / VA + 255) / 256;   // loads per thread per block
    static constexpr int NB = (RB * T / VBL + 255) / 256;
};

template <typename Te, int VE, int N, int T, int RB>
__device__ __forceinline__ void wgrad_fetch(u32x4 (&r)[N], const Te *__restrict__ src, uint32_t C,
                                            uint32_t col0, uint32_t row0, uint32_t row_end)
{
    constexpr uint32_t PER_ROW = T / VE;
#pragma unroll
    for (int n = 0; n < N; ++n) {
        const uint32_t v = threadIdx.x + 256u * (uint32_t)n;
        const uint32_t row = row0 + v / PER_ROW;
        r[n] = (u32x4){0u, 0u, 0u, 0u};
        if (v < (uint32_t)RB * PER_ROW && row < row_end)
            r[n] = *reinterpret_cast<const u32x4 *>(src + (size_t)row * C + col0 +
                                                    (v % PER_ROW) * VE);
    }
}

template <typename Te, int VE, int N, int T, int LDW, int RB>
__device__ __forceinline__ void wgrad_stage(float *lds, const u32x4 (&r)[N])
{
    constexpr uint32_t PER_ROW = T / VE;
#pragma unroll
    for (int n = 0; n < N; ++n) {
        const uint32_t v = threadIdx.x + 256u * (uint32_t)n;
        if (v >= (uint32_t)RB * PER_ROW) continue;
        float *dst = lds + (v / PER_ROW) * LDW + (v % PER_ROW) * VE;
        if constexpr (VE == 4) {
            *reinterpret_cast<f32x4 *>(dst) = __builtin_bit_cast(f32x4, r[n]);
        } else {   // eight bf16: widening is exact (the bits are the float's high half)
            const u32x4 u = r[n];
            *reinterpret_cast<f32x4 *>(dst) =
                (f32x4){__builtin_bit_cast(float, u.x << 16), __builtin_bit_cast(float, u.x & 0xffff0000u),
                        __builtin_bit_cast(float, u.y << 16), __builtin_bit_cast(float, u.y & 0xffff0000u)};
            *reinterpret_cast<f32x4 *>(dst + 4) =
                (f32x4){__builtin_bit_cast(float, u.z << 16), __builtin_bit_cast(float, u.z & 0xffff0000u),
                        __builtin_bit_cast(float, u.w << 16), __builtin_bit_cast(float, u.w & 0xffff0000u)};
        }
    }
}

// Eight k-slot values (two groups of four) for the 16x16x32 instruction.
// Three-term bf16 split of floats: v = hi + mid + lo + d with each term the
// nearest bf16 of what the previous ones leave (the differences are exact in
// float32) and |d| <= 2^-27 |v|.
__device__ __forceinline__ void split3_bf16x8(const f32x4 &z0, const f32x4 &z1, bf16x8 &hi,
                                              bf16x8 &mid, bf16x8 &lo)
{
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float z = e < 4 ? z0[e] : z1[e - 4];
        const __bf16 h = (__bf16)z;
        const float r1 = z - (float)h;
        const __bf16 m = (__bf16)r1;
        hi[e] = h;
        mid[e] = m;
        lo[e] = (__bf16)(r1 - (float)m);
    }
}

// bf16-origin values as bf16: their high halves, exactly.  (Whole vectors are
// bit-cast: a bit_cast of one ext-vector element reads element 0 in this
// toolchain.)
__device__ __forceinline__ bf16x8 bf16_exact8(const f32x4 &z0, const f32x4 &z1)
{
    const u32x4 u0 = __builtin_bit_cast(u32x4, z0), u1 = __builtin_bit_cast(u32x4, z1);
    const u32x4 o = {(u0[0] >> 16) | (u0[1] & 0xffff0000u), (u0[2] >> 16) | (u0[3] & 0xffff0000u),
                     (u1[0] >> 16) | (u1[1] & 0xffff0000u), (u1[2] >> 16) | (u1[3] & 0xffff0000u)};
    return __builtin_bit_cast(bf16x8, o);
}

// Partial blocks are stored as computed, rows of a by columns of b (a caller
// that passed B and A gets dW^T and transposes in the final sum).
template <typename Ta, typename Tb, int T>
__global__ void __launch_bounds__(256)
wgrad_mfma_kernel(const Ta *__restrict__ a, const Tb *__restrict__ b, float *__restrict__ part,
                  uint32_t rows, uint32_t rpc, int cb)
{
    using S = WgradShape<Ta, Tb, T>;
    constexpr int LDW = S::LDW, TQ = S::TQ;
    constexpr bool F32 = sizeof(Ta) == 4 && sizeof(Tb) == 4;
    constexpr bool SPLIT_A = sizeof(Ta) == 4 && !F32;   // a is the float operand
    constexpr bool SPLIT_B = sizeof(Tb) == 4 && !F32;
    __shared__ float sa[S::RB * LDW], sb[S::RB * LDW];
    const uint32_t C = 1u << cb;
    const uint32_t nside = C / (uint32_t)T;
    const uint32_t c0 = (blockIdx.x / nside) * T, d0 = (blockIdx.x % nside) * T;
    const uint32_t chunk = blockIdx.y;
    const uint32_t r_begin = chunk * rpc;
    const uint32_t r_end = min(rows, r_begin + rpc);
    const uint32_t lane = threadIdx.x & 63u, w = threadIdx.x >> 6;
    const uint32_t i = lane & 15u, q = lane >> 4;
    const bool active = T >= 32 || w == 0;
    const uint32_t tr0 = T >= 32 ? (w >> 1) * TQ : 0u, tc0 = T >= 32 ? (w & 1u) * TQ : 0u;
    f32x4 acc[TQ][TQ];
#pragma unroll
    for (int x = 0; x < TQ; ++x)
#pragma unroll
        for (int y = 0; y < TQ; ++y)
            acc[x][y] = (f32x4){0.0f, 0.0f, 0.0f, 0.0f};
    u32x4 ra[S::NA], rb[S::NB];
    wgrad_fetch<Ta, S::VA, S::NA, T, S::RB>(ra, a, C, c0, r_begin, r_end);
    wgrad_fetch<Tb, S::VBL, S::NB, T, S::RB>(rb, b, C, d0, r_begin, r_end);
    for (uint32_t r0 = r_begin; r0 < r_end; r0 += S::RB) {   // uniform over the workgroup
        __syncthreads();   // the previous block's readers are done
        wgrad_stage<Ta, S::VA, S::NA, T, LDW, S::RB>(sa, ra);
        wgrad_stage<Tb, S::VBL, S::NB, T, LDW, S::RB>(sb, rb);
        __syncthreads();
        if (r0 + S::RB < r_end) {
            wgrad_fetch<Ta, S::VA, S::NA, T, S::RB>(ra, a, C, c0, r0 + S::RB, r_end);
            wgrad_fetch<Tb, S::VBL, S::NB, T, S::RB>(rb, b, C, d0, r0 + S::RB, r_end);
        }
        if (!active)
            continue;
        if constexpr (F32) {
#pragma unroll 2
            for (int kb = 0; kb < S::RB; kb += 4) {
                const float *ra_ = sa + (kb + q) * LDW + i;
                const float *rb_ = sb + (kb + q) * LDW + i;
                float av[TQ], bv[TQ];
#pragma unroll
                for (int x = 0; x < TQ; ++x)
                    av[x] = ra_[16 * (tr0 + x)];
#pragma unroll
                for (int y = 0; y < TQ; ++y)
                    bv[y] = rb_[16 * (tc0 + y)];
#pragma unroll
                for (int x = 0; x < TQ; ++x)
#pragma unroll
                    for (int y = 0; y < TQ; ++y)
                        acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[x], bv[y], acc[x][y],
                                                                        0, 0, 0);
            }
        } else {
#pragma unroll 1
            for (int kb = 0; kb < S::RB; kb += 32) {
                // the float operand's three terms, the bf16 operand's one;
                // k-slot e of lane (i, q) is row kb + q + 4e
                constexpr int NSA = SPLIT_A ? 3 : 1, NSB = SPLIT_B ? 3 : 1;
                bf16x8 av[NSA][TQ], bv[NSB][TQ];
#pragma unroll
                for (int x = 0; x < TQ; ++x) {
                    const float *src = sa + (kb + q) * LDW + 16 * (tr0 + x) + i;
                    const f32x4 z0 = {src[0], src[4 * LDW], src[8 * LDW], src[12 * LDW]};
                    const f32x4 z1 = {src[16 * LDW], src[20 * LDW], src[24 * LDW], src[28 * LDW]};
                    if constexpr (SPLIT_A)
                        split3_bf16x8(z0, z1, av[0][x], av[1][x], av[2][x]);
                    else
                        av[0][x] = bf16_exact8(z0, z1);
                }
#pragma unroll
                for (int y = 0; y < TQ; ++y) {
                    const float *src = sb + (kb + q) * LDW + 16 * (tc0 + y) + i;
                    const f32x4 z0 = {src[0], src[4 * LDW], src[8 * LDW], src[12 * LDW]};
                    const f32x4 z1 = {src[16 * LDW], src[20 * LDW], src[24 * LDW], src[28 * LDW]};
                    if constexpr (SPLIT_B)
                        split3_bf16x8(z0, z1, bv[0][y], bv[1][y], bv[2][y]);
                    else
                        bv[0][y] = bf16_exact8(z0, z1);
                }
#pragma unroll
                for (int x = 0; x < TQ; ++x)
#pragma unroll
                    for (int y = 0; y < TQ; ++y)
#pragma unroll
                        for (int t = 0; t < NSA * NSB; ++t)
                            acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                av[t % NSA][x], bv[t / NSA][y], acc[x][y], 0, 0, 0);
            }
        }
    }
    if (!active)
        return;
    // lane 16q + j of a tile holds its rows 4q + r (channels of a) of column j
    float *out = part + (size_t)chunk * C * C;
#pragma unroll
    for (int x = 0; x < TQ; ++x)
#pragma unroll
        for (int y = 0; y < TQ; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t row = c0 + 16u * (tr0 + x) + 4u * q + r;
                const uint32_t col = d0 + 16u * (tc0 + y) + i;
                out[(size_t)row * C + col] = acc[x][y][r];
            }
}

// The same for C < 16 on the VALU: one thread per output of one chunk.
template <typename Ta, typename Tb>
__global__ void __launch_bounds__(256)
wgrad_valu_kernel(const Ta *__restrict__ a, const Tb *__restrict__ b, float *__restrict__ part,
                  uint32_t rows, uint32_t rpc, int cb)
{
    const uint32_t C = 1u << cb;
    const uint32_t o = threadIdx.x;
    if (o >= C * C) return;
    const uint32_t ci = o >> cb, cj = o & (C - 1u);
    const uint32_t chunk = blockIdx.x;
    const uint32_t r_end = min(rows, chunk * rpc + rpc);
    float acc = 0.0f;
    for (uint32_t r = chunk * rpc; r < r_end; ++r)
        acc = fmaf(to_f(a[(size_t)r * C + ci]), to_f(b[(size_t)r * C + cj]), acc);
    part[(size_t)chunk * C * C + o] = acc;
}

// out[g][i] = sum over the chunks c of group g = blockIdx.y (ascending, at
// most `group` of them) of part[c][i]; with one group this is the total.
// tcb > 0: part holds C x C matrices (C = 2^tcb) and out gets the transposed
// sum.  Eight loads are issued before their adds (in the same ascending
// order), so a thread waits for one memory round trip per eight chunks, not
// per chunk.
constexpr uint32_t kSumThreads = 64;
__global__ void __launch_bounds__(kSumThreads)
sum_partials_kernel(const float *__restrict__ part, float *__restrict__ out, uint32_t n,
                    uint32_t chunks, uint32_t group, uint32_t tcb)
{
    const uint32_t i = blockIdx.x * kSumThreads + threadIdx.x;
    if (i >= n) return;
    const uint32_t c0 = blockIdx.y * group;
    const uint32_t c1 = min(chunks, c0 + group);
    float s = 0.0f;
    uint32_t c = c0;
    for (; c + 8u <= c1; c += 8u) {
        float v[8];
#pragma unroll
        for (uint32_t j = 0; j < 8u; ++j)
            v[j] = part[(size_t)(c + j) * n + i];
#pragma unroll
        for (uint32_t j = 0; j < 8u; ++j)
            s += v[j];
    }
    for (; c < c1; ++c)
        s += part[(size_t)c * n + i];
    const uint32_t o = tcb ? ((i & ((1u << tcb) - 1u)) << tcb) | (i >> tcb) : i;
    out[(size_t)blockIdx.y * n + o] = s;
}

template <typename T>
hipError_t launch_pack_b(const T *w, T *p, int cb, bool trans, hipStream_t st)
{
    const uint32_t n = 1u << (2 * cb);
    hipLaunchKernelGGL((pack_b_kernel<T>), dim3((n + 255u) / 256u), dim3(256), 0, st, w, p, cb,
                       trans ? 1 : 0);
    return hipGetLastError();
}

template <typename Tin, typename Tout, typename T, int CB>
hipError_t launch_project_mfma(const Tin *in, const T *wpk, Tout *out, uint32_t rows,
                               hipStream_t st)
{
    using PC = ProjCols<T, CB>;
    const uint32_t slices = PC::C / PC::NCOL;
    const uint32_t nblk = (rows + 63u) / 64u;
    uint32_t gx = 512u / slices;
    gx = gx < 1u ? 1u : (gx > nblk ? nblk : gx);
    hipLaunchKernelGGL((project_mfma_kernel<Tin, Tout, T, CB>), dim3(gx, slices), dim3(256), 0,
                       st, in, wpk, out, rows);
    return hipGetLastError();
}

// out = in W (TRANS: in W^T); wpk is W (or W^T) packed, wraw the raw matrix.
template <typename Tin, typename Tout, typename T, bool TRANS>
hipError_t project(const Tin *in, const T *wpk, const T *wraw, Tout *out, uint32_t rows, int cb,
                   hipStream_t st)
{
    if (rows == 0) return hipSuccess;
    switch (cb) {
#define WHTMIX_PJ_CASE(c) \
    case c:               \
        if constexpr (ProjCols<T, c>::OK) return launch_project_mfma<Tin, Tout, T, c>(in, wpk, out, rows, st); \
        break;
        WHTMIX_PJ_CASE(5) WHTMIX_PJ_CASE(6) WHTMIX_PJ_CASE(7) WHTMIX_PJ_CASE(8)
        WHTMIX_PJ_CASE(9) WHTMIX_PJ_CASE(10) WHTMIX_PJ_CASE(11) WHTMIX_PJ_CASE(12)
#undef WHTMIX_PJ_CASE
    default: break;
    }
    const uint64_t total = (uint64_t)rows << cb;
    hipLaunchKernelGGL((project_rows_kernel<Tin, Tout, T, TRANS>),
                       dim3((uint32_t)((total + 255u) / 256u)), dim3(256), 0, st, in, wraw, out,
                       total, cb);
    return hipGetLastError();
}

template <typename Ta, typename Tb>
hipError_t wgrad(const Ta *a, const Tb *b, float *part, float *out, uint32_t rows, int cb,
                 hipStream_t st)
{
    const uint32_t C = 1u << cb;
    const WgradPlan wp = wgrad_plan(rows, cb);
    // A float a against a bf16 b runs on the matrix cores as (b, a), whose sum
    // is transposed at the end: the kernel with the bf16 operand first keeps
    // fewer registers (two workgroups per CU at T = 128 instead of one).
    constexpr bool SWAP = sizeof(Ta) == 4 && sizeof(Tb) == 2;
    const bool swapped = SWAP && C >= 16;
    if (wp.chunks == 0) {
        // no rows: sum_partials over zero chunks writes zeros
    } else if (C >= 16) {
        using T1 = std::conditional_t<SWAP, Tb, Ta>;
        using T2 = std::conditional_t<SWAP, Ta, Tb>;
        const T1 *p1 = reinterpret_cast<const T1 *>(SWAP ? (const void *)b : (const void *)a);
        const T2 *p2 = reinterpret_cast<const T2 *>(SWAP ? (const void *)a : (const void *)b);
        const uint32_t T = C < 128u ? C : 128u;
        const dim3 grid((C / T) * (C / T), wp.chunks);
        if (T == 16)
            hipLaunchKernelGGL((wgrad_mfma_kernel<T1, T2, 16>), grid, dim3(256), 0, st, p1,
                               p2, part, rows, wp.rows_per_chunk, cb);
        else if (T == 32)
            hipLaunchKernelGGL((wgrad_mfma_kernel<T1, T2, 32>), grid, dim3(256), 0, st, p1,
                               p2, part, rows, wp.rows_per_chunk, cb);
        else if (T == 64)
            hipLaunchKernelGGL((wgrad_mfma_kernel<T1, T2, 64>), grid, dim3(256), 0, st, p1,
                               p2, part, rows, wp.rows_per_chunk, cb);
        else
            hipLaunchKernelGGL((wgrad_mfma_kernel<T1, T2, 128>), grid, dim3(256), 0, st, p1,
                               p2, part, rows, wp.rows_per_chunk, cb);
    } else {
        hipLaunchKernelGGL((wgrad_valu_kernel<Ta, Tb>), dim3(wp.chunks), dim3(256), 0, st, a, b,
                           part, rows, wp.rows_per_chunk, cb);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // fixed-order sum: groups of consecutive chunks, then the groups
    const uint32_t n = C * C, nb = (n + kSumThreads - 1u) / kSumThreads;
    const uint32_t tcb = swapped ? (uint32_t)cb : 0u;
    if (wp.chunks <= kWgradGroup) {
        hipLaunchKernelGGL(sum_partials_kernel, dim3(nb), dim3(kSumThreads), 0, st, part, out, n,
                           wp.chunks, kWgradGroup, tcb);
        return hipGetLastError();
    }
    float *gsum = part + (size_t)wp.chunks * n;
    hipLaunchKernelGGL(sum_partials_kernel, dim3(nb, wp.groups()), dim3(kSumThreads), 0, st, part,
                       gsum, n, wp.chunks, kWgradGroup, 0u);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(sum_partials_kernel, dim3(nb), dim3(kSumThreads), 0, st, gsum, out, n,
                       wp.groups(), wp.groups(), tcb);
    return hipGetLastError();
}

// The block's backward with its projections fused into the mixer backward's
// passes (module_backward_fused decides when):
//   OUTER_FWD of Z = X W_in and dZ' = dY W_out^T, matrix-core prologues, one
//   launch -> the backward's middle phase: dG, and both Z and dZ' through the
//   gain up to their last pass, in place in wsx and wsd                 [1]
//   -> OUTER_INV of wsx -> Z' (float32); dW_out = Z'^T dY                 [2]
//   -> OUTER_INV of wsd with the epilogue: dZ (float32) and dX = dZ W_in^T;
//      dW_in = X^T dZ                                                     [3]
// Z and dZ' never reach memory: they exist only as the outer transforms.
template <typename T, int K, int CB>
hipError_t module_backward_fused_k(const ModuleBackwardArgs &m)
{
    constexpr Split sp = module_split(K);
    constexpr int A = sp.A, HB = sp.HB, R = sp.R;
    static_assert(A == three_pass_split(K).A && R == three_pass_split(K).R,
                  "the backward's middle phase runs the mixer's split");
    const hipStream_t st = m.stream;
    const uint32_t rows = (uint32_t)(((uint64_t)m.B * m.nvalid) >> CB);
    const uint32_t CC = 1u << (2 * CB);
    const T *x = static_cast<const T *>(m.x);
    const T *dy = static_cast<const T *>(m.dy);
    const T *w_in = static_cast<const T *>(m.w_in);
    T *pk = static_cast<T *>(m.wpack);
    T *p_in = pk, *p_out_t = pk + CC, *p_in_te = pk + 2 * CC;
    const PackJobs<T> jobs{{w_in, static_cast<const T *>(m.w_out), w_in},
                           {p_in, p_out_t, p_in_te},
                           {PACK_PROLOGUE, PACK_PROLOGUE_T, PACK_EPILOGUE_T}};
    if constexpr (Proj<T, CB>::X32)
        hipLaunchKernelGGL(pack_x32_kernel, dim3((CC + 255u) / 256u), dim3(256), 0, st, jobs, CB);
    else
        hipLaunchKernelGGL((pack_std_kernel<T>), dim3((CC + 255u) / 256u), dim3(256), 0, st, jobs,
                           CB);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = record(m.events[0], st)) != hipSuccess) return e;
    const bool separable = m.gain_kind == GAIN_LOG_SEPARABLE;
    const BackwardLayout lay =
        backward_layout(PLAN_THREE_PASS, K, m.B, int64_t(1) << CB, separable);
    float *wsx = m.bwd_ws + lay.wsx;
    float *wsd = m.bwd_ws + lay.wsd;
    hipLaunchKernelGGL((module_outer_fwd2_kernel<A, HB, R, T, CB>),
                       dim3((uint32_t)(2 * (m.B << HB))), dim3(1u << (A - VB)), 0, st, x, p_in,
                       dy, p_out_t, wsx, wsd, m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    BackwardArgs g{};
    g.gain_kind = m.gain_kind;
    g.gain = m.gain;
    g.gain_t = m.gain_t;
    g.gain_c = m.gain_c;
    g.dgain = m.dgain;
    g.dgt = m.dgt;
    g.dgc = m.dgc;
    g.cbits = CB;
    g.ws = m.bwd_ws;
    g.B = m.B;
    g.K = K;
    g.nvalid = m.nvalid;
    g.dtype = DTYPE_F32;
    g.plan = PLAN_THREE_PASS;
    g.stream = st;
    if ((e = launch_backward_middle(g)) != hipSuccess) return e;
    if ((e = record(m.events[1], st)) != hipSuccess) return e;
    if ((e = launch_outer_inv<K, float>(wsx, m.zp, m.B, m.nvalid, st)) != hipSuccess) return e;
    if ((e = wgrad<float, T>(m.zp, dy, m.wpart, m.dw_out, rows, CB, st)) != hipSuccess) return e;
    if ((e = record(m.events[2], st)) != hipSuccess) return e;
    // dZ (float32, for dW_in) and dX = dZ W_in^T from one pass over wsd
    hipLaunchKernelGGL((module_outer_inv_kernel<A, HB, R, T, CB, true>),
                       dim3((uint32_t)(m.B << HB)), dim3(1u << (A - VB)), 0, st, wsd, p_in_te,
                       static_cast<T *>(m.dx), m.dzp, m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = wgrad<T, float>(x, m.dzp, m.wpart, m.dw_in, rows, CB, st)) != hipSuccess) return e;
    return record(m.events[3], st);
}

// The same for bf16 C = 256 on the 2^16 outer tiles (pair_split, which is the
// mixer's split, and so the backward middle phase's, from 2^26 elements).
template <int K>
hipError_t module_backward_fused_pair(const ModuleBackwardArgs &m)
{
    constexpr Split sp = pair_split(K);
    constexpr int HB = sp.HB, R = sp.R;
    static_assert(K >= 26 && sp.A == three_pass_split(K).A && R == three_pass_split(K).R,
                  "the backward's middle phase runs the mixer's split");
    using T = __bf16;
    constexpr int CB = kPairCB;
    const hipStream_t st = m.stream;
    const uint32_t rows = (uint32_t)(((uint64_t)m.B * m.nvalid) >> CB);
    const uint32_t CC = 1u << (2 * CB);
    const T *x = static_cast<const T *>(m.x);
    const T *dy = static_cast<const T *>(m.dy);
    const T *w_in = static_cast<const T *>(m.w_in);
    T *pk = static_cast<T *>(m.wpack);
    T *p_in = pk, *p_out_t = pk + CC, *p_in_te = pk + 2 * CC;
    const PackX32Jobs jobs{{w_in, static_cast<const T *>(m.w_out), w_in},
                           {p_in, p_out_t, p_in_te},
                           {PACK_PROLOGUE, PACK_PROLOGUE_T, PACK_EPILOGUE_T}};
    hipLaunchKernelGGL(pack_x32_kernel, dim3((CC + 255u) / 256u), dim3(256), 0, st, jobs, CB);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if ((e = record(m.events[0], st)) != hipSuccess) return e;
    const bool separable = m.gain_kind == GAIN_LOG_SEPARABLE;
    const BackwardLayout lay = backward_layout(PLAN_THREE_PASS, K, m.B, kPairC, separable);
    float *wsx = m.bwd_ws + lay.wsx;
    float *wsd = m.bwd_ws + lay.wsd;
    hipLaunchKernelGGL((module_outer_fwd2_pair_kernel<HB, R>), dim3((uint32_t)(2 * (m.B << HB))),
                       dim3(kPairThreads), 0, st, x, p_in, dy, p_out_t, wsx, wsd, m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    BackwardArgs g{};
    g.gain_kind = m.gain_kind;
    g.gain = m.gain;
    g.gain_t = m.gain_t;
    g.gain_c = m.gain_c;
    g.dgain = m.dgain;
    g.dgt = m.dgt;
    g.dgc = m.dgc;
    g.cbits = CB;
    g.ws = m.bwd_ws;
    g.B = m.B;
    g.K = K;
    g.nvalid = m.nvalid;
    g.dtype = DTYPE_F32;
    g.plan = PLAN_THREE_PASS;
    g.stream = st;
    if ((e = launch_backward_middle(g)) != hipSuccess) return e;
    if ((e = record(m.events[1], st)) != hipSuccess) return e;
    if ((e = launch_outer_inv<K, float>(wsx, m.zp, m.B, m.nvalid, st)) != hipSuccess) return e;
    if ((e = wgrad<float, T>(m.zp, dy, m.wpart, m.dw_out, rows, CB, st)) != hipSuccess) return e;
    if ((e = record(m.events[2], st)) != hipSuccess) return e;
    hipLaunchKernelGGL((module_outer_inv_pair_kernel<HB, R, true>), dim3((uint32_t)(m.B << HB)),
                       dim3(kPairThreads), 0, st, wsd, p_in_te, static_cast<T *>(m.dx), m.dzp,
                       m.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = wgrad<T, float>(x, m.dzp, m.wpart, m.dw_in, rows, CB, st)) != hipSuccess) return e;
    return record(m.events[3], st);
}

template <typename T, int CB>
hipError_t module_backward_fused_cb(const ModuleBackwardArgs &m)
{
    switch (m.K) {
#define WHTMIX_MB_CASE(k) \
    case k: return module_backward_fused_k<T, k, CB>(m);
        WHTMIX_MB_CASE(12) WHTMIX_MB_CASE(13) WHTMIX_MB_CASE(14) WHTMIX_MB_CASE(15)
        WHTMIX_MB_CASE(16) WHTMIX_MB_CASE(17) WHTMIX_MB_CASE(18) WHTMIX_MB_CASE(19)
        WHTMIX_MB_CASE(20) WHTMIX_MB_CASE(21) WHTMIX_MB_CASE(22) WHTMIX_MB_CASE(23)
        WHTMIX_MB_CASE(24) WHTMIX_MB_CASE(25)
#undef WHTMIX_MB_CASE
    default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t module_backward(const ModuleBackwardArgs &m)
{
    const bool want_dg = m.gain_kind == GAIN_LOG_SEPARABLE ? (m.dgt != nullptr)
                                                           : (m.dgain != nullptr);
    if (want_dg && m.B > 0 && ((uint64_t)m.B << m.K) / 16u <= 0xffffffffull &&
        module_backward_fused(m.plan, m.cbits, m.dtype, m.K)) {
        switch (m.cbits) {
        case 4: return module_backward_fused_cb<T, 4>(m);
        case 5: return module_backward_fused_cb<T, 5>(m);
        case 6: return module_backward_fused_cb<T, 6>(m);
        case 7: return module_backward_fused_cb<T, 7>(m);
        case kPairCB:
            if constexpr (!std::is_same<T, __bf16>::value) break;
            switch (m.K) {
            case 26: return module_backward_fused_pair<26>(m);
            case 27: return module_backward_fused_pair<27>(m);
            case 28: return module_backward_fused_pair<28>(m);
            default: break;
            }
            break;
        default: break;
        }
    }
    const hipStream_t st = m.stream;
    const int cb = m.cbits;
    const uint32_t rows = (uint32_t)(((uint64_t)m.B * m.nvalid) >> cb);
    const size_t CC = (size_t)1 << (2 * cb);
    const T *x = static_cast<const T *>(m.x);
    const T *dy = static_cast<const T *>(m.dy);
    const T *w_in = static_cast<const T *>(m.w_in);
    const T *w_out = static_cast<const T *>(m.w_out);
    T *pk = static_cast<T *>(m.wpack);
    T *p_in = pk, *p_out_t = pk + CC, *p_in_t = pk + 2 * CC;
    hipError_t e;
    if (cb >= 4) {   // matrix-core projections need the packed forms
        if ((e = launch_pack_b<T>(w_in, p_in, cb, false, st)) != hipSuccess) return e;
        if ((e = launch_pack_b<T>(w_out, p_out_t, cb, true, st)) != hipSuccess) return e;
        if ((e = launch_pack_b<T>(w_in, p_in_t, cb, true, st)) != hipSuccess) return e;
    }
    if ((e = record(m.events[0], st)) != hipSuccess) return e;
    // Z = X W_in, Z' = mixer(Z)
    if ((e = project<T, float, T, false>(x, p_in, w_in, m.z, rows, cb, st)) != hipSuccess) return e;
    LaunchArgs a{};
    a.x = m.z;
    a.y = m.zp;
    a.gain_kind = m.gain_kind;
    a.gain = m.gain;
    a.gain_t = m.gain_t;
    a.gain_c = m.gain_c;
    a.cbits = cb;
    a.ws = m.mix_ws;
    a.B = m.B;
    a.K = m.K;
    a.nvalid = m.nvalid;
    a.dtype = DTYPE_F32;
    a.plan = m.plan;
    a.stream = st;
    if (m.B > 0 && (e = launch(a)) != hipSuccess) return e;
    // dZ' = dY W_out^T, dW_out = Z'^T dY
    if ((e = project<T, float, T, true>(dy, p_out_t, w_out, m.dzp, rows, cb, st)) != hipSuccess)
        return e;
    if ((e = wgrad<float, T>(m.zp, dy, m.wpart, m.dw_out, rows, cb, st)) != hipSuccess) return e;
    if ((e = record(m.events[1], st)) != hipSuccess) return e;
    // the mixer's gradients at (Z, dZ'): dZ in place of dZ', and the gain's
    BackwardArgs g{};
    g.x = m.z;
    g.dy = m.dzp;
    g.dx = m.dzp;
    g.gain_kind = m.gain_kind;
    g.gain = m.gain;
    g.gain_t = m.gain_t;
    g.gain_c = m.gain_c;
    g.dgain = m.dgain;
    g.dgt = m.dgt;
    g.dgc = m.dgc;
    g.cbits = cb;
    g.ws = m.bwd_ws;
    g.B = m.B;
    g.K = m.K;
    g.nvalid = m.nvalid;
    g.dtype = DTYPE_F32;
    g.plan = m.plan;
    g.stream = st;
    if ((e = launch_backward(g)) != hipSuccess) return e;
    if ((e = record(m.events[2], st)) != hipSuccess) return e;
    // dX = dZ W_in^T, dW_in = X^T dZ
    if ((e = project<float, T, T, true>(m.dzp, p_in_t, w_in, static_cast<T *>(m.dx), rows, cb,
                                        st)) != hipSuccess)
        return e;
    if ((e = wgrad<T, float>(x, m.dzp, m.wpart, m.dw_in, rows, cb, st)) != hipSuccess) return e;
    return record(m.events[3], st);
}
}  // namespace

hipError_t launch_module(const ModuleArgs &m)
{
    if (m.dtype == DTYPE_BF16)
        return dispatch_module_gain<__bf16>(m);
    return dispatch_module_gain<float>(m);
}

hipError_t launch_module_backward(const ModuleBackwardArgs &m)
{
    if (m.dtype == DTYPE_BF16)
        return module_backward<__bf16>(m);
    return module_backward<float>(m);
}

}  // namespace whtmix
