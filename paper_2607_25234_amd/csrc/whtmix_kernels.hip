// WHTMix forward kernels for gfx950 (MI355X).
//
// One slice of the mixer (section III-B, eqs. (2)-(3), joint gain G[N][C]) is
//     y = (1/L) H_L (g o H_L x),   L = N*C = 2^K,
// on the flattened row-major index f = n*C + c (whtmix_plan.h explains why).
// The Walsh-Hadamard transform is add/subtract work: no multiplies except the
// single gain product, and it is bound by memory traffic and VALU issue, not
// by matrix throughput, so there is no MFMA here.
//
// The tile machinery (layouts, butterflies, LDS exchanges, memory access,
// gains) and the OUTER_FWD / OUTER_INV kernels, which the backward pass
// shares, are in whtmix_tile.h.
//
// Kernels:
//   FUSED     whole slice in one tile: forward over all bits, gain, inverse.
//   OUTER_FWD contiguous 2^A chunk of x: forward over its A bits, stored to
//             the workspace in runs of 2^R so each middle tile is contiguous.
//   MIDDLE    one 2^HB x 2^R workspace tile (or one run in a group of
//             slices): forward over the HB high bits, gain, inverse over the
//             HB bits (R low bits carried along).
//   OUTER_INV mirror of OUTER_FWD: inverse over the A low bits, store y.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "whtmix_launch.h"
#include "whtmix_plan.h"
#include "whtmix_tile.h"

namespace whtmix {
namespace {

using namespace tile;

// ---------------------------------------------------------------- kernels
// x and y hold `nvalid` = N*C elements per slice (N real tokens); the
// transform runs over the zero-padded slice of 2^K = N_pad*C elements.

// FUSED: tile = whole slice (M = K), one workgroup per slice b.
template <int K, typename T, class Gain>
__global__ void __launch_bounds__(1 << (K - VB))
fused_kernel(const T *__restrict__ x, T *__restrict__ y, Gain gain, uint32_t nvalid)
{
    using G = Groups<K, 0>;
    __shared__ float lds[pad(1u << K)];
    const uint32_t tau = threadIdx.x;
    const size_t base = (size_t)blockIdx.x * nvalid;
    float v[V], gv[V];
    load_tile<G::TOP, K, T>(v, x + base, nvalid, tau);
    gain.template load<G::SL, ContigMap>(gv, 0, tau);
    butterflies<G::JT, VB>(v);
    forward_groups<K, 0, 0, G::TOP>(lds, v, tau);
    apply_gain<K>(v, gv);
    if constexpr (G::NBOT > 0)
        inverse_groups<K, 0, G::NBOT - 1>(lds, v, tau);
    butterflies<G::JT, VB>(v);
    store_tile<G::TOP, K, T>(v, y + base, nvalid, tau);
}

// FUSED for 2^16 elements: one 1024-thread workgroup holds the slice as two
// 2^15 register sets (set = tile bit 15).  Bit 15 is a register butterfly
// between the sets, right after the load and right before the store; bits
// 0..14 run the 2^15 schedule on each set in turn through the same LDS.  The
// gain of the second set is read when the first set is done with its own.
template <typename T, class Gain>
__global__ void __launch_bounds__(1 << (15 - VB))
fused_pair_kernel(const T *__restrict__ x, T *__restrict__ y, Gain gain, uint32_t nvalid)
{
    constexpr int K = 16, M = 15;
    using G = Groups<M, 0>;
    __shared__ float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const size_t base = (size_t)blockIdx.x * nvalid;
    const uint32_t valid0 = min(nvalid, 1u << M);
    const uint32_t valid1 = nvalid > (1u << M) ? nvalid - (1u << M) : 0u;
    float v0[V], v1[V];
    load_tile<G::TOP, M, T>(v0, x + base, valid0, tau);
    load_tile<G::TOP, M, T>(v1, x + base + (1u << M), valid1, tau);
    cross_butterflies(v0, v1);
    butterflies<0, VB>(v0);
    butterflies<0, VB>(v1);
    forward_groups<M, 0, 0, G::TOP>(lds, v0, tau);
    forward_groups<M, 0, 0, G::TOP, true>(lds, v1, tau);
    {
        float gv[V];
        gain.template load<G::SL, ContigMap>(gv, 0, tau);
        apply_gain<K>(v0, gv);
    }
    inverse_groups<M, 0, G::NBOT - 1>(lds, v0, tau);
    butterflies<0, VB>(v0);
    {
        float gv[V];
        gain.template load<G::SL, ContigMap>(gv, 1u << M, tau);
        apply_gain<K>(v1, gv);
    }
    inverse_groups<M, 0, G::NBOT - 1>(lds, v1, tau);
    butterflies<0, VB>(v1);
    cross_butterflies(v0, v1);
    store_tile<G::TOP, M, T>(v0, y + base, valid0, tau);
    store_tile<G::TOP, M, T>(v1, y + base + (1u << M), valid1, tau);
}

// MIDDLE: logical tile = run * B + b (the B slices sharing a gain tile are
// adjacent); workgroups are renumbered so adjacent logical tiles land on the
// same XCD (blocks are dealt round-robin over the 8 XCDs) and share its L2.
template <int A, int HB, int R, class Gain>
__global__ void __launch_bounds__(1 << (HB + R - VB))
middle_kernel(float *__restrict__ ws, Gain gain, uint32_t nslices)
{
    constexpr int M = HB + R;
    using G = Groups<M, R>;
    __shared__ float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t nblk = gridDim.x;
    uint32_t logical = blockIdx.x;
    if ((nblk & 7u) == 0)
        logical = (blockIdx.x & 7u) * (nblk >> 3) + (blockIdx.x >> 3);
    const uint32_t run = logical / nslices;
    const size_t b = logical - run * nslices;
    const __amdgpu_buffer_rsrc_t tile =
        buffer(ws + (b << (A + HB)) + ((size_t)run << M), (1u << M) * 4u);
    float v[V], gv[V];
    load_layout<G::TOP, ContigMap, float>(v, tile, tau);
    gain.template load<G::SL, GainMap<A, R>, true>(gv, run << R, tau);
    butterflies<G::JT, VB>(v);
    forward_groups<M, R, 0, G::TOP>(lds, v, tau);
    apply_gain<A + HB>(v, gv);
    if constexpr (G::NBOT > 0)
        inverse_groups<M, R, G::NBOT - 1>(lds, v, tau);
    butterflies<G::JT, VB>(v);
    store_layout<G::TOP, ContigMap, float>(v, tile, tau);
}

// MIDDLE over slice groups (nb > 1, middle_slices_per_group): workgroup w
// reads the gain of run w mod 2^(A-R) once and takes that run in slices
// (w >> (A-R)) * nb .. + nb - 1 one after the other, each slice's tile
// loaded after the previous one is stored.  Consecutive workgroups take
// consecutive runs; the blocks sharing a run's gain are 2^(A-R) apart, a
// multiple of 8, so on one XCD.  Measured on 4 slices of 2^23 (nb = 4):
// 48.9 us against 51.3 us for middle_kernel; the XCD renumbering of
// middle_kernel measured 51.2 us here, and prefetching the next slice's tile
// into registers 50.4 us.  The first tile's loads go out before the gain's
// (49.0 against 50.0 us, averaged with cold calls).
template <int A, int HB, int R, class Gain>
__global__ void __launch_bounds__(1 << (HB + R - VB))
middle_group_kernel(float *__restrict__ ws, Gain gain, uint32_t nb)
{
    constexpr int M = HB + R;
    using G = Groups<M, R>;
    __shared__ float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t run = blockIdx.x & ((1u << (A - R)) - 1u);
    float *const base = ws + (((size_t)(blockIdx.x >> (A - R)) * nb) << (A + HB)) +
                        ((size_t)run << M);
    float v[V], gv[V];
    load_layout<G::TOP, ContigMap, float>(v, buffer(base, (1u << M) * 4u), tau);
    gain.template load<G::SL, GainMap<A, R>, true>(gv, run << R, tau);   // needed later
#pragma unroll 1
    for (uint32_t j = 0; j < nb; ++j) {
        butterflies<G::JT, VB>(v);
        forward_groups<M, R, 0, G::TOP, true>(lds, v, tau);
        apply_gain<A + HB>(v, gv);
        if constexpr (G::NBOT > 0)
            inverse_groups<M, R, G::NBOT - 1>(lds, v, tau);
        butterflies<G::JT, VB>(v);
        store_layout<G::TOP, ContigMap, float>(
            v, buffer(base + ((size_t)j << (A + HB)), (1u << M) * 4u), tau);
        if (j + 1 < nb)
            load_layout<G::TOP, ContigMap, float>(
                v, buffer(base + ((size_t)(j + 1) << (A + HB)), (1u << M) * 4u), tau);
    }
}

__device__ __forceinline__ float to_float(float v) { return v; }
__device__ __forceinline__ float to_float(__bf16 v) { return (float)v; }
template <typename T>
__device__ __forceinline__ T from_float(float v) { return (T)v; }   // bf16: round to nearest even

// SMALL: 2^K <= 2^10; one 256-thread workgroup per slice, every stage on the
// LDS copy.
template <typename T, class Gain>
__global__ void __launch_bounds__(256)
small_kernel(const T *__restrict__ x, T *__restrict__ y, Gain gain, int K, uint32_t nvalid)
{
    __shared__ float s[1 << kMaxSmall];
    const int L = 1 << K;
    const size_t base = (size_t)blockIdx.x * nvalid;
    const float scale = 1.0f / (float)L;
    for (int i = threadIdx.x; i < L; i += blockDim.x)
        s[i] = (uint32_t)i < nvalid ? to_float(x[base + i]) : 0.0f;
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
    for (int i = threadIdx.x; i < (int)nvalid; i += blockDim.x)
        y[base + i] = from_float<T>(s[i]);
}

// ---------------------------------------------------------------- launchers
inline hipError_t record(hipEvent_t ev, hipStream_t st)
{
    return ev ? hipEventRecord(ev, st) : hipSuccess;
}

template <int K, typename T, class Gain>
hipError_t launch_fused(const T *x, T *y, Gain gain, const LaunchArgs &a)
{
    hipError_t e = record(a.events[0], a.stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((fused_kernel<K, T, Gain>), dim3((uint32_t)a.B), dim3(1u << (K - VB)), 0,
                       a.stream, x, y, gain, a.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(a.events[1], a.stream);
}

template <typename T, class Gain>
hipError_t launch_fused_pair(const T *x, T *y, Gain gain, const LaunchArgs &a)
{
    hipError_t e = record(a.events[0], a.stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((fused_pair_kernel<T, Gain>), dim3((uint32_t)a.B), dim3(1u << (15 - VB)), 0,
                       a.stream, x, y, gain, a.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(a.events[1], a.stream);
}

template <int A, int HB, int R, class Gain>
hipError_t launch_middle_split(const LaunchArgs &a, Gain gain)
{
    static_assert(HB >= 1 && HB + R >= kMinTile && HB + R <= kMaxTile, "middle tile size");
    const long long nb = middle_slices_per_group(a.B, A - R, HB + R - VB);
    return with_forward_middle_gain(gain, a.B, A + HB, [&](auto g) {
        if (nb > 1)
            hipLaunchKernelGGL((middle_group_kernel<A, HB, R, decltype(g)>),
                               dim3((uint32_t)((a.B / nb) << (A - R))), dim3(1u << (HB + R - VB)),
                               0, a.stream, a.ws, g, (uint32_t)nb);
        else
            hipLaunchKernelGGL((middle_kernel<A, HB, R, decltype(g)>),
                               dim3((uint32_t)(a.B << (A - R))), dim3(1u << (HB + R - VB)), 0,
                               a.stream, a.ws, g, (uint32_t)a.B);
        return hipGetLastError();
    });
}

template <int K, typename T, class Gain>
hipError_t launch_three_pass(const T *x, T *y, Gain gain, const LaunchArgs &a)
{
    constexpr Split sp = three_pass_split(K);
    constexpr int A = sp.A, HB = sp.HB, R = sp.R;
    static_assert(A >= kMinTile && A <= kMaxOuter, "outer tile size");
    static_assert(HB + R >= kMinTile && HB + R <= kMaxTile, "middle tile size");
    static_assert(HB >= 1 && R >= 0 && R <= A, "split");
    const hipStream_t st = a.stream;
    hipError_t e = record(a.events[0], st);
    if (e != hipSuccess) return e;
    if ((e = launch_outer_fwd<K, T>(x, a.ws, a.B, a.nvalid, st)) != hipSuccess) return e;
    if ((e = record(a.events[1], st)) != hipSuccess) return e;
    if ((e = launch_middle_split<A, HB, R>(a, gain)) != hipSuccess) return e;
    if ((e = record(a.events[2], st)) != hipSuccess) return e;
    if ((e = launch_outer_inv<K, T>(a.ws, y, a.B, a.nvalid, st)) != hipSuccess) return e;
    return record(a.events[3], st);
}

template <typename T, class Gain>
hipError_t launch_small(const T *x, T *y, Gain gain, const LaunchArgs &a)
{
    hipError_t e = record(a.events[0], a.stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((small_kernel<T, Gain>), dim3((uint32_t)a.B), dim3(256), 0, a.stream, x, y,
                       gain, a.K, a.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(a.events[1], a.stream);
}

template <typename T, class Gain>
hipError_t dispatch(const LaunchArgs &a, Gain gain)
{
    const T *x = static_cast<const T *>(a.x);
    T *y = static_cast<T *>(a.y);
    if (a.plan == PLAN_SMALL)
        return launch_small<T, Gain>(x, y, gain, a);
    if (a.plan == PLAN_FUSED) {
        switch (a.K) {
#define WHTMIX_FUSED_CASE(k) \
    case k: return launch_fused<k, T, Gain>(x, y, gain, a);
            WHTMIX_FUSED_CASE(11) WHTMIX_FUSED_CASE(12) WHTMIX_FUSED_CASE(13)
            WHTMIX_FUSED_CASE(14) WHTMIX_FUSED_CASE(15)
#undef WHTMIX_FUSED_CASE
        case kMaxFused: return launch_fused_pair<T, Gain>(x, y, gain, a);
        default: return hipErrorInvalidValue;
        }
    }
    switch (a.K) {
#define WHTMIX_3P_CASE(k) \
    case k: return launch_three_pass<k, T, Gain>(x, y, gain, a);
        WHTMIX_3P_CASE(12) WHTMIX_3P_CASE(13) WHTMIX_3P_CASE(14) WHTMIX_3P_CASE(15)
        WHTMIX_3P_CASE(16) WHTMIX_3P_CASE(17) WHTMIX_3P_CASE(18) WHTMIX_3P_CASE(19)
        WHTMIX_3P_CASE(20) WHTMIX_3P_CASE(21) WHTMIX_3P_CASE(22) WHTMIX_3P_CASE(23)
        WHTMIX_3P_CASE(24) WHTMIX_3P_CASE(25) WHTMIX_3P_CASE(26) WHTMIX_3P_CASE(27)
        WHTMIX_3P_CASE(28) WHTMIX_3P_CASE(29) WHTMIX_3P_CASE(30)
#undef WHTMIX_3P_CASE
    default: return hipErrorInvalidValue;
    }
}


template <int K, class Gain>
hipError_t launch_middle_k(const LaunchArgs &a, Gain gain)
{
    if constexpr (K >= kPairModuleMinK) {
        constexpr Split sp = pair_split(K);
        if (a.pair_outer)
            return launch_middle_split<sp.A, sp.HB, sp.R, Gain>(a, gain);
    }
    if (a.pair_outer)
        return hipErrorInvalidValue;
    constexpr Split sp = module_split(K);
    return launch_middle_split<sp.A, sp.HB, sp.R, Gain>(a, gain);
}

template <class Gain>
hipError_t dispatch_middle(const LaunchArgs &a, Gain gain)
{
    switch (a.K) {
#define WHTMIX_MID_CASE(k) \
    case k: return launch_middle_k<k, Gain>(a, gain);
        WHTMIX_MID_CASE(12) WHTMIX_MID_CASE(13) WHTMIX_MID_CASE(14) WHTMIX_MID_CASE(15)
        WHTMIX_MID_CASE(16) WHTMIX_MID_CASE(17) WHTMIX_MID_CASE(18) WHTMIX_MID_CASE(19)
        WHTMIX_MID_CASE(20) WHTMIX_MID_CASE(21) WHTMIX_MID_CASE(22) WHTMIX_MID_CASE(23)
        WHTMIX_MID_CASE(24) WHTMIX_MID_CASE(25) WHTMIX_MID_CASE(26) WHTMIX_MID_CASE(27)
        WHTMIX_MID_CASE(28) WHTMIX_MID_CASE(29) WHTMIX_MID_CASE(30)
#undef WHTMIX_MID_CASE
    default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t dispatch_gain(const LaunchArgs &a)
{
    if (a.gain_kind == GAIN_LOG_SEPARABLE)
        return dispatch<T>(a, LogSeparableGain{a.gain_t, a.gain_c, (uint32_t)a.cbits});
    return dispatch<T>(a, FullGain{a.gain});
}

}  // namespace

hipError_t launch_middle(const LaunchArgs &a)
{
    if (a.gain_kind == GAIN_LOG_SEPARABLE)
        return dispatch_middle(a, LogSeparableGain{a.gain_t, a.gain_c, (uint32_t)a.cbits});
    return dispatch_middle(a, FullGain{a.gain});
}

hipError_t launch(const LaunchArgs &a)
{
    if (a.dtype == DTYPE_BF16)
        return dispatch_gain<__bf16>(a);
    return dispatch_gain<float>(a);
}

}  // namespace whtmix
