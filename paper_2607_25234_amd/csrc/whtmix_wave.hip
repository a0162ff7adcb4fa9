// Wave tiles: the three passes of slices of 2^12 .. 2^16 elements on
// one-wave tiles of 2^9 elements whose butterflies stay inside the wave
// (gfx950).  Three plans run them:
//   WAVE_TILES  three launches, one tile per workgroup; AUTO takes it for up
//               to 3 slices of 2^16 elements (image1k: 9.2 -> 7.3 us per call
//               against THREE_PASS);
//   TWO_PASS    a fold pass in place of the first two launches (below), then
//               the third; AUTO takes it for up to 48 slices of 2^15 and 4-16
//               of 2^16;
//   ONE_LAUNCH  all three passes in a single cooperative launch, ordered by
//               per-slice completion counters (forced only: slower).
//
// The mixer of one slice is y = (1/L) H_L (g o H_L x) on the flat index
// f = n*C + c, L = N_pad*C = 2^K (the channel and token transforms of section
// III-B, eqs. (2)-(3), are one Walsh-Hadamard transform over the K bits of f;
// whtmix_plan.h), run as three passes: forward over the 9 low bits of f,
// forward over the HB = K-9 high bits + gain + inverse over them, inverse over
// the low bits.
//
// Tiles.  A workgroup is one wave; a tile is 2^9 elements, 8 per lane.  Every
// butterfly stays inside the wave, with no LDS:
//   - register bits: butterflies between a lane's own registers;
//   - lane bits 0..3: DPP (quad_perm for bits 0-1; row_shl / row_shr by 4
//     or 8 with bank masks for bits 2-3) fetches the partner's value, and one
//     fma with the lane's sign (+1 low partner, -1 high partner) forms
//     a + b or a - b exactly (multiplying by +-1 is exact);
//   - lane bits 4, 5: v_permlane16_swap / v_permlane32_swap exchange a lane
//     bit with register bit 2 (a 2x2 transpose of register pairs), the
//     butterfly runs between registers, and a second swap restores the
//     layout.
// Layouts (t = tile-local element index, k = register, lambda = lane):
//   V4 (16-byte float32 groups): t = (k & 3) | lambda << 2 | (k >> 2) << 8
//   V8 (16-byte bf16 groups):    t = k | lambda << 3
// x and y move in their element type's layout; the float32 workspace always
// moves in 16-byte groups of 4 consecutive elements.
//
// Passes (R = 9 - HB, the run of contiguous low elements the middle pass
// carries untransformed; K <= 16 gives R >= 2, so a 4-group never straddles
// a run):
//   1. tile (b, hi) = x[b][hi*2^9 ...]: forward over its 9 bits, stored to the
//      workspace as runs: element t goes to (t >> R)*2^9 + hi*2^R + (t mod 2^R).
//   2. tile (b, run) = workspace[b][run*2^9 ...] (u = hi*2^R + e): forward over
//      u's HB high bits, times G[f] * 2^-K at f = hi*2^9 + run*2^R + e, inverse
//      over the same bits, stored in place.
//   3. tile (b, hi): gathered from the runs, inverse over its 9 bits, stored to
//      y with round to nearest even for bf16.
//
// ONE_LAUNCH scheduling.  The grid is launched cooperatively (every workgroup
// resident).  Workgroup w takes tiles w, w + P, w + 2P, ... of each pass in
// turn.  Counter c0[b] (c1[b]) counts finished pass-1 (pass-2) tiles of slice
// b; a pass-2 (pass-3) tile of slice b starts once it reaches 2^HB.  The
// smallest unfinished tile never waits on anything unfinished, and its
// workgroup is resident and working on it, so the schedule always completes.
// Each wait is bounded: after `spin_limit` polls it raises the call's error
// word and every later wait gives up at once, so every wave exits.  The last
// workgroup to exit (it counts exits) folds the call's error word into a
// sticky word that the host reads, and returns all counters to zero for the
// next call.  Memory ordering: a finished tile's stores are released to agent
// scope by the counter increment (all lanes' stores complete first); a wait
// ends with an agent-scope acquire fence before the tile's loads.  A
// cooperative launch alone costs about 20 us, and such a hand-off costs more
// than a kernel boundary, which is why AUTO never picks it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "whtmix_launch.h"
#include "whtmix_plan.h"
#include "whtmix_tile.h"

namespace whtmix {
namespace wave {

constexpr int TB = 9;    // tile bits
constexpr int NV = 8;    // values per lane

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- wave butterflies
template <int J>
__device__ __forceinline__ void reg_bfly(float (&v)[NV])
{
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        if (!(k & (1 << J))) {
            const float a = v[k], b = v[k | (1 << J)];
            v[k] = a + b;
            v[k | (1 << J)] = a - b;
        }
    }
}

// Value of lane (lambda ^ 2^J), J in 0..3, by DPP.
template <int J>
__device__ __forceinline__ float lane_partner(float x)
{
    const int xi = __builtin_bit_cast(int, x);
    int p;
    if constexpr (J == 0) {
        p = __builtin_amdgcn_update_dpp(0, xi, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
    } else if constexpr (J == 1) {
        p = __builtin_amdgcn_update_dpp(0, xi, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
    } else if constexpr (J == 2) {
        // lanes with bit 2 set (banks 1, 3 of each row) read lambda - 4
        // (row_shr:4); the others (banks 0, 2) read lambda + 4 (row_shl:4)
        const int hi = __builtin_amdgcn_update_dpp(0, xi, 0x114, 0xF, 0xA, false);
        p = __builtin_amdgcn_update_dpp(hi, xi, 0x104, 0xF, 0x5, false);
    } else {
        // bit 3: banks 2, 3 read lambda - 8 (row_shr:8), banks 0, 1 lambda + 8
        const int hi = __builtin_amdgcn_update_dpp(0, xi, 0x118, 0xF, 0xC, false);
        p = __builtin_amdgcn_update_dpp(hi, xi, 0x108, 0xF, 0x3, false);
    }
    return __builtin_bit_cast(float, p);
}

// Butterfly over lane bit J (0..3): the low lane of a pair gets a + b, the
// high lane a - b (a: the low lane's value).
template <int J>
__device__ __forceinline__ void lane_bfly(float (&v)[NV], uint32_t lane)
{
    const float s = (lane & (1u << J)) ? -1.0f : 1.0f;
#pragma unroll
    for (int k = 0; k < NV; ++k)
        v[k] = __builtin_fmaf(s, v[k], lane_partner<J>(v[k]));
}

// Exchange lane bit 5 (W = 32) or 4 (W = 16) with register bit 2 for every
// register pair (k, k + 4): an involution.
template <int W>
__device__ __forceinline__ void swap_k2(float (&v)[NV])
{
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const unsigned a = __builtin_bit_cast(unsigned, v[k]);
        const unsigned b = __builtin_bit_cast(unsigned, v[k + 4]);
        if constexpr (W == 32) {
            const auto r = __builtin_amdgcn_permlane32_swap(a, b, false, false);
            v[k] = __builtin_bit_cast(float, (unsigned)r[0]);
            v[k + 4] = __builtin_bit_cast(float, (unsigned)r[1]);
        } else {
            const auto r = __builtin_amdgcn_permlane16_swap(a, b, false, false);
            v[k] = __builtin_bit_cast(float, (unsigned)r[0]);
            v[k + 4] = __builtin_bit_cast(float, (unsigned)r[1]);
        }
    }
}

// Butterflies over lane bits [J0, 6) and register bit 2.
template <int J0>
__device__ __forceinline__ void wave_bfly(float (&v)[NV], uint32_t lane)
{
    reg_bfly<2>(v);
    if constexpr (J0 <= 0) lane_bfly<0>(v, lane);
    if constexpr (J0 <= 1) lane_bfly<1>(v, lane);
    if constexpr (J0 <= 2) lane_bfly<2>(v, lane);
    if constexpr (J0 <= 3) lane_bfly<3>(v, lane);
    if constexpr (J0 <= 4) {
        swap_k2<16>(v);
        reg_bfly<2>(v);
        swap_k2<16>(v);
    }
    swap_k2<32>(v);
    reg_bfly<2>(v);
    swap_k2<32>(v);
}

// All 9 bits of a tile (any layout: every register and lane bit).
__device__ __forceinline__ void wht9(float (&v)[NV], uint32_t lane)
{
    reg_bfly<0>(v);
    reg_bfly<1>(v);
    wave_bfly<0>(v, lane);
}

// ---------------------------------------------------------------- layouts
// First element t of 16-byte group g (registers 4g .. 4g+3) of lane lambda.
template <int ELT>
__device__ __forceinline__ uint32_t group_t(uint32_t lane, int g)
{
    if constexpr (ELT == 4)
        return (lane << 2) | ((uint32_t)g << 8);   // V4
    else
        return (lane << 3) | ((uint32_t)g << 2);   // V8
}

// Workspace offset of outer-tile element t (relative to slice base + hi*2^R).
template <int R>
__device__ __forceinline__ uint32_t run_off(uint32_t t)
{
    return ((t >> R) << TB) | (t & ((1u << R) - 1u));
}

__device__ __forceinline__ void ld4(float (&v)[NV], int g, const float *p)
{
    const f32x4 q = *reinterpret_cast<const f32x4 *>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e)
        v[4 * g + e] = q[e];
}

__device__ __forceinline__ void st4(const float (&v)[NV], int g, float *p)
{
    const f32x4 q = {v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]};
    *reinterpret_cast<f32x4 *>(p) = q;
}

// x tile (2^9 elements, `valid` of them real) into registers, in the element
// type's layout.  valid is a multiple of the 16-byte group (host-checked).
template <typename T>
__device__ __forceinline__ void load_x(float (&v)[NV], const T *src, uint32_t valid,
                                       uint32_t lane)
{
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const uint32_t t0 = group_t<4>(lane, g);
            if (t0 < valid) {
                ld4(v, g, reinterpret_cast<const float *>(src) + t0);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) v[4 * g + e] = 0.0f;
            }
        }
    } else {
        const uint32_t t0 = lane << 3;
        if (t0 < valid) {
            const u32x4 q = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4 *>(src + t0));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t wv = q[e];
                v[2 * e] = __builtin_bit_cast(float, wv << 16);
                v[2 * e + 1] = __builtin_bit_cast(float, wv & 0xffff0000u);
            }
        } else {
#pragma unroll
            for (int k = 0; k < NV; ++k) v[k] = 0.0f;
        }
    }
}

template <typename T>
__device__ __forceinline__ void store_y(const float (&v)[NV], T *dst, uint32_t valid,
                                        uint32_t lane)
{
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            const uint32_t t0 = group_t<4>(lane, g);
            if (t0 < valid)
                st4(v, g, reinterpret_cast<float *>(dst) + t0);
        }
    } else {
        const uint32_t t0 = lane << 3;
        if (t0 < valid) {
            u32x4 q;
#pragma unroll
            for (int e = 0; e < 4; ++e) {   // round to nearest even, two per word
                const uint32_t lo = __builtin_bit_cast(unsigned short, (__bf16)v[2 * e]);
                const uint32_t hi = __builtin_bit_cast(unsigned short, (__bf16)v[2 * e + 1]);
                q[e] = lo | (hi << 16);
            }
            *reinterpret_cast<u32x4 *>(dst + t0) = q;
        }
    }
}

// ---------------------------------------------------------------- gains
// Four consecutive gains from frequency f0 (a multiple of 4).
template <class Gain>
struct Gain4;

template <bool NT>
struct Gain4<tile::FullGainT<NT>> {
    __device__ static __forceinline__ void load(const tile::FullGainT<NT> &gn, float (&gv)[NV],
                                                int g, uint32_t f0)
    {
        const f32x4 *p = reinterpret_cast<const f32x4 *>(gn.g + f0);
        const f32x4 q = NT ? __builtin_nontemporal_load(p) : *p;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            gv[4 * g + e] = q[e];
    }
};

template <>
struct Gain4<tile::LogSeparableGain> {
    __device__ static __forceinline__ void load(const tile::LogSeparableGain &gn,
                                                float (&gv)[NV], int g, uint32_t f0)
    {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            gv[4 * g + e] = gn.at(f0 + e);
    }
};

// Gains of middle tile `run` in the V4 layout (u = hi*2^R + e).
template <int R, class Gain>
__device__ __forceinline__ void load_gain(const Gain &gn, float (&gv)[NV], uint32_t run,
                                          uint32_t lane)
{
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        const uint32_t u0 = group_t<4>(lane, g);
        const uint32_t f0 = ((u0 >> R) << TB) | (run << R) | (u0 & ((1u << R) - 1u));
        Gain4<Gain>::load(gn, gv, g, f0);
    }
}

// ---------------------------------------------------------------- counters
struct Counters {
    uint32_t *c0;        // [B] finished pass-1 tiles per slice
    uint32_t *c1;        // [B] finished pass-2 tiles per slice
    uint32_t *exited;    // workgroups past their last counter access
    uint32_t *call_err;  // raised by a wait that ran out of polls
    uint32_t *sticky;    // errors of past calls, read and cleared by the host
};

// Block layout: c0 at [0, B), c1 at [B, 2B); the three single words at the
// end of the kCounterWords block (the host reads the sticky word there).
__device__ __forceinline__ Counters counters(uint32_t *ctr, uint32_t B)
{
    return Counters{ctr, ctr + B, ctr + kCounterWords - 3, ctr + kCounterWords - 2,
                    ctr + kCounterWords - 1};
}

// The tile's stores are complete (every lane's) before the increment is
// visible at agent scope.
__device__ __forceinline__ void signal_done(uint32_t *c)
{
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait for *c >= target; false when this call has failed.
__device__ __forceinline__ bool wait_for(const uint32_t *c, uint32_t target, uint32_t *call_err,
                                         uint32_t spin_limit)
{
    uint32_t polls = 0;
    bool ok = true;
    while (__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (__hip_atomic_load(call_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) {
            ok = false;
            break;
        }
        if (++polls > spin_limit) {
            __hip_atomic_store(call_err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ok = false;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return ok;
}

// ---------------------------------------------------------------- pass tiles
// The three passes on one tile each (shared by both plans).  Slice bits K,
// HB = K - 9 high bits, R = 9 - HB carried run bits.
template <int K>
struct Shape {
    static constexpr int HB = K - TB;
    static constexpr int R = TB - HB;
    static_assert(HB >= 3 && R >= 2, "wave tiles cover 2^12 .. 2^16 elements per slice");
    static constexpr uint32_t TILES = 1u << HB;   // tiles per slice and pass
};

__device__ __forceinline__ uint32_t tile_valid9(uint32_t nvalid, uint32_t hi)
{
    const uint32_t start = hi << TB;
    return nvalid <= start ? 0u : min(nvalid - start, 1u << TB);
}

// Pass 1: tile (b, hi) of x, forward over its 9 bits, stored as runs.
template <int K, typename T>
__device__ __forceinline__ void pass1_tile(const T *__restrict__ x, float *__restrict__ ws,
                                           uint32_t b, uint32_t hi, uint32_t nvalid,
                                           uint32_t lane)
{
    using S = Shape<K>;
    float v[NV];
    load_x<T>(v, x + (size_t)b * nvalid + (hi << TB), tile_valid9(nvalid, hi), lane);
    wht9(v, lane);
    float *dst = ws + ((size_t)b << K) + (hi << S::R);
#pragma unroll
    for (int g = 0; g < 2; ++g)
        st4(v, g, dst + run_off<S::R>(group_t<sizeof(T)>(lane, g)));
}

// Pass 2: tile (b, run) of the workspace, forward over the HB high bits,
// times the gain (gv, already gathered) and 2^-K, inverse; in place.
template <int K>
__device__ __forceinline__ void pass2_tile(float *__restrict__ ws, const float (&gv)[NV],
                                           uint32_t b, uint32_t run, uint32_t lane)
{
    using S = Shape<K>;
    constexpr float scale = 1.0f / (float)(1u << K);   // exact power of two
    float *tile = ws + ((size_t)b << K) + (run << TB);
    float v[NV];
#pragma unroll
    for (int g = 0; g < 2; ++g)
        ld4(v, g, tile + group_t<4>(lane, g));
    wave_bfly<S::R - 2>(v, lane);
#pragma unroll
    for (int k = 0; k < NV; ++k)
        v[k] *= gv[k] * scale;
    wave_bfly<S::R - 2>(v, lane);
#pragma unroll
    for (int g = 0; g < 2; ++g)
        st4(v, g, tile + group_t<4>(lane, g));
}

// Pass 3: tile (b, hi) gathered from the runs, inverse over its 9 bits,
// stored to y (nothing for a tile wholly in the padding).
template <int K, typename T>
__device__ __forceinline__ void pass3_tile(const float *__restrict__ ws, T *__restrict__ y,
                                           uint32_t b, uint32_t hi, uint32_t nvalid,
                                           uint32_t lane)
{
    using S = Shape<K>;
    const uint32_t valid = tile_valid9(nvalid, hi);
    if (valid == 0)
        return;   // uniform per workgroup
    const float *src = ws + ((size_t)b << K) + (hi << S::R);
    float v[NV];
#pragma unroll
    for (int g = 0; g < 2; ++g)
        ld4(v, g, src + run_off<S::R>(group_t<sizeof(T)>(lane, g)));
    wht9(v, lane);
    store_y<T>(v, y + (size_t)b * nvalid + (hi << TB), valid, lane);
}

// ---------------------------------------------------------------- WAVE_TILES
// Three launches, one tile per workgroup: tile i = b * 2^HB + (hi or run).
// The runs are 2^R floats (16 bytes at R = 2), so the 2^(5-R) neighbouring
// tiles whose runs share a 128-byte line of the workspace (passes 1 and 3) or
// of the gain (pass 2) are numbered onto one XCD (tile::outer_block): each
// line is then written back or fetched once, by one L2, not once per XCD.
template <int K>
__device__ __forceinline__ uint32_t wave_tile()
{
    return tile::outer_block<Shape<K>::R>(blockIdx.x, gridDim.x);
}

template <int K, typename T>
__global__ void __launch_bounds__(64)
wave_pass1_kernel(const T *__restrict__ x, float *__restrict__ ws, uint32_t nvalid)
{
    using S = Shape<K>;
    const uint32_t i = wave_tile<K>();
    pass1_tile<K, T>(x, ws, i >> S::HB, i & (S::TILES - 1u), nvalid, threadIdx.x);
}

template <int K, class Gain>
__global__ void __launch_bounds__(64)
wave_pass2_kernel(float *__restrict__ ws, Gain gain)
{
    using S = Shape<K>;
    const uint32_t i = wave_tile<K>();
    const uint32_t run = i & (S::TILES - 1u);
    float gv[NV];
    load_gain<S::R>(gain, gv, run, threadIdx.x);
    pass2_tile<K>(ws, gv, i >> S::HB, run, threadIdx.x);
}

template <int K, typename T>
__global__ void __launch_bounds__(64)
wave_pass3_kernel(const float *__restrict__ ws, T *__restrict__ y, uint32_t nvalid)
{
    using S = Shape<K>;
    const uint32_t i = wave_tile<K>();
    pass3_tile<K, T>(ws, y, i >> S::HB, i & (S::TILES - 1u), nvalid, threadIdx.x);
}

// ---------------------------------------------------------------- ONE_LAUNCH
template <int K, typename T, class Gain>
__global__ void __launch_bounds__(64)
one_launch_kernel(const T *__restrict__ x, T *__restrict__ y, Gain gain, float *__restrict__ ws,
                  uint32_t *ctr, uint32_t B, uint32_t nvalid, uint32_t spin_limit)
{
    using S = Shape<K>;
    constexpr int HB = S::HB;
    constexpr uint32_t TILES = S::TILES;
    const uint32_t lane = threadIdx.x;
    const uint32_t P = gridDim.x;
    const uint32_t ntiles = B << HB;
    const Counters cn = counters(ctr, B);

    // Gain of this workgroup's first middle tile, read before any waiting.
    float gv[NV];
    if (blockIdx.x < ntiles)
        load_gain<S::R>(gain, gv, blockIdx.x & (TILES - 1u), lane);

    // Pass 1: forward over the 9 low bits of f, stored as runs.
    for (uint32_t i = blockIdx.x; i < ntiles; i += P) {
        const uint32_t b = i >> HB;
        pass1_tile<K, T>(x, ws, b, i & (TILES - 1u), nvalid, lane);
        signal_done(cn.c0 + b);
    }

    // Pass 2: forward over the HB high bits, gain, inverse; in place.
    bool ok = true;
    for (uint32_t i = blockIdx.x; ok && i < ntiles; i += P) {
        const uint32_t b = i >> HB, run = i & (TILES - 1u);
        if (i != blockIdx.x)
            load_gain<S::R>(gain, gv, run, lane);
        ok = wait_for(cn.c0 + b, TILES, cn.call_err, spin_limit);
        if (!ok) break;
        pass2_tile<K>(ws, gv, b, run, lane);
        signal_done(cn.c1 + b);
    }

    // Pass 3: inverse over the 9 low bits, stored to y.
    for (uint32_t i = blockIdx.x; ok && i < ntiles; i += P) {
        const uint32_t b = i >> HB;
        ok = wait_for(cn.c1 + b, TILES, cn.call_err, spin_limit);
        if (!ok) break;
        pass3_tile<K, T>(ws, y, b, i & (TILES - 1u), nvalid, lane);
    }

    // Exit: the last workgroup out resets the counters for the next call.
    __syncthreads();
    if (lane == 0) {
        const uint32_t prior =
            __hip_atomic_fetch_add(cn.exited, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        if (prior == P - 1u) {
            const uint32_t e =
                __hip_atomic_load(cn.call_err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (e)
                __hip_atomic_fetch_or(cn.sticky, e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (uint32_t j = 0; j < 2 * B; ++j)
                __hip_atomic_store(ctr + j, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(cn.call_err, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(cn.exited, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// ---------------------------------------------------------------- TWO_PASS
// Two launches for slices of 2^15 and 2^16 elements: a fold pass that
// replaces passes 1 and 2, then pass 3 as above.
//
// Write t9 = mu*2^Q + j for the 9 low bits of f (Q = 21 - K low bits j, the
// A = 9 - Q bits mu above them) and hi for the HB high bits.  H_2^9 is
// H_2^A (on mu) times H_2^Q (on j), so the forward transform over the low
// bits, read at one value m of mu, is
//   u[hi][m*2^Q + j] = H_2^Q( sum_a (-1)^popcount(m & a) x[hi][a*2^Q + .] )[j]:
// a signed sum of the 2^A blocks of 2^Q elements of row hi, then a
// transform of length 2^Q.  Workgroup (b, m) evaluates it for all 2^HB rows
// from the whole slice (read 2^(9-Q) times over, once per workgroup, from
// L2), so it holds the 2^12 elements (hi, j) with mu = m fully transformed
// over the low bits.  It then runs the forward over hi, the gain, the
// inverse over hi, and stores its elements to the workspace in the run
// layout that pass 3 gathers (8 whole middle tiles, 16 contiguous KiB).
// One launch boundary fewer than WAVE_TILES, at the price of each workgroup
// reading the whole slice.
//
// 512 threads, 8 values each, in two register layouts:
//   M1: j = (t mod 2^LJ) << 2 | k mod 4, hi = t >> LJ | (k >> 2) << (HB - 1);
//   M2: j = t mod 2^Q, hi = (h mod 2^W0) | k << W0 | (h >> W0) << (HB - 1),
//       h = t >> Q;
// with LJ = Q - 2 lane bits of j and W0 = 6 - LJ lane bits of hi in M1.  M1
// holds j's low bits in registers and lanes (the fold's 16-byte groups,
// H_2^Q by registers and DPP) and hi's bits except the three wave bits
// [W0, W0 + 3) in lanes (DPP, permlane swaps) and register bit 2; M2 holds
// those three wave bits in registers.  The layouts meet in a 16 KiB LDS
// array in natural [hi][j] order (M1 writes 16-byte rows of a wave's 1 KiB,
// M2 reads 64 consecutive floats per register: no bank conflicts).
template <int K>
struct Fold {
    static constexpr int HB = K - TB;     // high bits of f
    static constexpr int R = TB - HB;     // workspace run bits (pass 3's layout)
    static constexpr int Q = 21 - K;      // low bits a workgroup keeps
    static constexpr int A = TB - Q;      // folded bits: 2^A workgroups per slice
    static constexpr int LJ = Q - 2;      // lane bits of j in M1
    static constexpr int W0 = 6 - LJ;     // lane bits of hi in M1
    static_assert((K == 15 || K == 16) && HB == W0 + 4 && R >= 2 && Q - R == 3,
                  "the fold pass covers 2^15- and 2^16-element slices");
};

__device__ __forceinline__ float fold_sign(uint32_t m, uint32_t a)
{
    return (__builtin_popcount(m & a) & 1) ? -1.0f : 1.0f;
}

// Four consecutive x elements at byte offset voff + soff of the slice's
// buffer resource, as float32.  The resource spans the slice's valid
// elements, so groups past them (padded N; whole groups, as nvalid is a
// multiple of 8) read as zeros, with no branch: every load of the fold is
// issued before the first is waited for.  Temporal: the slice is read by
// every workgroup of its fold and stays in L2.
template <typename T>
__device__ __forceinline__ f32x4 load_x4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff)
{
    if constexpr (sizeof(T) == 4) {
        return __builtin_bit_cast(
            f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, tile::kTemporal));
    } else {
        typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 q = __builtin_bit_cast(
            u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, tile::kTemporal));
        return f32x4{__builtin_bit_cast(float, q[0] << 16),
                     __builtin_bit_cast(float, q[0] & 0xffff0000u),
                     __builtin_bit_cast(float, q[1] << 16),
                     __builtin_bit_cast(float, q[1] & 0xffff0000u)};
    }
}

// Workgroups are dealt to the 8 XCDs round-robin (block i on XCD i mod 8), so
// block i takes slice b = (i >> (A + 3)) * 8 + i mod 8, part m = (i >> 3) mod
// 2^A: the 2^A workgroups of a slice share one XCD, whose L2 fetches the
// slice for all of them (32 slices of 2^15: 9.9 -> 8.9 us per call against
// the plain numbering).  The grid covers B rounded up to a multiple of 8;
// blocks past the last slice exit at once.
template <int K, typename T, class Gain>
__global__ void __launch_bounds__(512)
fold_pass_kernel(const T *__restrict__ x, float *__restrict__ ws, Gain gain, uint32_t nvalid,
                 uint32_t nslices)
{
    using F = Fold<K>;
    constexpr int HB = F::HB, Q = F::Q, LJ = F::LJ, W0 = F::W0;
    constexpr float scale = 1.0f / (float)(1u << K);   // exact power of two
    __shared__ __attribute__((aligned(16))) float lds[1u << (HB + Q)];

    const uint32_t t = threadIdx.x, lane = t & 63u;
    const uint32_t b = ((blockIdx.x >> (F::A + 3)) << 3) | (blockIdx.x & 7u);
    const uint32_t m = (blockIdx.x >> 3) & ((1u << F::A) - 1u);
    if (b >= nslices)
        return;   // uniform per workgroup, before any barrier

    // M2 coordinates and this workgroup's gains (read first, used last).
    const uint32_t j2 = t & ((1u << Q) - 1u), h2 = t >> Q;
    auto hi2 = [&](int k) {
        return (h2 & ((1u << W0) - 1u)) | ((uint32_t)k << W0) | ((h2 >> W0) << (HB - 1));
    };
    float gv[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k)
        gv[k] = gain.at((hi2(k) << TB) | (m << Q) | j2) * scale;

    // M1 coordinates.
    const uint32_t j1 = (t & ((1u << LJ) - 1u)) << 2;
    const uint32_t h1 = t >> LJ;   // hi without its top bit (register bit 2)

    // Fold: the signed sum over a of the blocks of row hi, then H over j.
    constexpr uint32_t EB = sizeof(T);
    const __amdgpu_buffer_rsrc_t xr = tile::buffer(x + (size_t)b * nvalid, nvalid * EB);
    const uint32_t voff = ((h1 << TB) | j1) * EB;
    // Workgroup m starts at block m and wraps: the 2^A workgroups of a slice
    // read different lines at any moment, so each line misses in L2 once.
    float v[NV];
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
        const uint32_t row = ((uint32_t)rr << (HB - 1 + TB)) * EB;
        f32x4 acc = load_x4<T>(xr, voff, row + (m << Q) * EB) * fold_sign(m, m);
#pragma unroll
        for (uint32_t i = 1; i < (1u << F::A); ++i) {
            const uint32_t a = (m + i) & ((1u << F::A) - 1u);
            acc += fold_sign(m, a) * load_x4<T>(xr, voff, row + (a << Q) * EB);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[4 * rr + e] = acc[e];
    }
    reg_bfly<0>(v);
    reg_bfly<1>(v);
    lane_bfly<0>(v, lane);
    lane_bfly<1>(v, lane);
    lane_bfly<2>(v, lane);
    if constexpr (LJ == 4)
        lane_bfly<3>(v, lane);

    // Forward over hi: its lane bits and top bit here, its wave bits in M2.
    wave_bfly<LJ>(v, lane);
#pragma unroll
    for (int rr = 0; rr < 2; ++rr)
        st4(v, rr, lds + (((h1 | ((uint32_t)rr << (HB - 1))) << Q) | j1));
    __syncthreads();
    float u[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k)
        u[k] = lds[(hi2(k) << Q) | j2];
    reg_bfly<0>(u);
    reg_bfly<1>(u);
    reg_bfly<2>(u);
#pragma unroll
    for (int k = 0; k < NV; ++k)
        u[k] *= gv[k];
    reg_bfly<0>(u);
    reg_bfly<1>(u);
    reg_bfly<2>(u);
    // Each thread writes back the words it read: no barrier between.
#pragma unroll
    for (int k = 0; k < NV; ++k)
        lds[(hi2(k) << Q) | j2] = u[k];
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < 2; ++rr)
        ld4(v, rr, lds + (((h1 | ((uint32_t)rr << (HB - 1))) << Q) | j1));
    wave_bfly<LJ>(v, lane);

    // Store in pass 3's run layout: t9 -> (t9 >> R) << 9 | hi << R | t9 mod 2^R.
    const uint32_t t9 = (m << Q) | j1;
    float *dst = ws + ((size_t)b << K) + ((t9 >> F::R) << TB) + (t9 & ((1u << F::R) - 1u));
#pragma unroll
    for (int rr = 0; rr < 2; ++rr)
        st4(v, rr, dst + ((h1 | ((uint32_t)rr << (HB - 1))) << F::R));
}

// ---------------------------------------------------------------- launch
inline hipError_t record(hipEvent_t ev, hipStream_t st)
{
    return ev ? hipEventRecord(ev, st) : hipSuccess;
}

template <int K, typename T, class Gain>
hipError_t launch_one_launch_k(const LaunchArgs &a, Gain gain)
{
    auto kern = one_launch_kernel<K, T, Gain>;
    const uint32_t ntiles = (uint32_t)a.B << Shape<K>::HB;
    // Every workgroup must be resident: at most the device's resident count.
    static thread_local int cached_dev = -1, cached_max = 0;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (cached_dev != dev) {
        int per_cu = 0, cus = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, 64, 0);
        if (e != hipSuccess) return e;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        cached_dev = dev;
        cached_max = per_cu * cus;
    }
    const uint32_t grid = (uint32_t)std::min<int64_t>((int64_t)ntiles, (int64_t)cached_max);
    if (grid == 0) return hipErrorInvalidConfiguration;
    const T *x = static_cast<const T *>(a.x);
    T *y = static_cast<T *>(a.y);
    float *ws = a.ws;
    uint32_t *ctr = a.counters;
    uint32_t B = (uint32_t)a.B, nvalid = a.nvalid, spin = a.spin_limit;
    void *args[] = {&x, &y, &gain, &ws, &ctr, &B, &nvalid, &spin};
    if ((e = record(a.events[0], a.stream)) != hipSuccess) return e;
    e = hipLaunchCooperativeKernel(reinterpret_cast<const void *>(kern), dim3(grid), dim3(64),
                                   args, 0, a.stream);
    if (e != hipSuccess) return e;
    return record(a.events[1], a.stream);
}

template <int K, typename T, class Gain>
hipError_t launch_wave_tiles_k(const LaunchArgs &a, Gain gain)
{
    const dim3 grid((uint32_t)a.B << Shape<K>::HB), block(64);
    const T *x = static_cast<const T *>(a.x);
    T *y = static_cast<T *>(a.y);
    const hipStream_t st = a.stream;
    hipError_t e = record(a.events[0], st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((wave_pass1_kernel<K, T>), grid, block, 0, st, x, a.ws, a.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = record(a.events[1], st)) != hipSuccess) return e;
    hipLaunchKernelGGL((wave_pass2_kernel<K, Gain>), grid, block, 0, st, a.ws, gain);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = record(a.events[2], st)) != hipSuccess) return e;
    hipLaunchKernelGGL((wave_pass3_kernel<K, T>), grid, block, 0, st, a.ws, y, a.nvalid);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return record(a.events[3], st);
}

template <int K, typename T, class Gain>
hipError_t launch_two_pass_k(const LaunchArgs &a, Gain gain)
{
    if constexpr (K == 15 || K == 16) {
        const T *x = static_cast<const T *>(a.x);
        T *y = static_cast<T *>(a.y);
        const hipStream_t st = a.stream;
        hipError_t e = record(a.events[0], st);
        if (e != hipSuccess) return e;
        const uint32_t groups = (uint32_t)((a.B + 7) / 8);   // of 8 slices, one per XCD
        hipLaunchKernelGGL((fold_pass_kernel<K, T, Gain>), dim3(groups << (Fold<K>::A + 3)),
                           dim3(512), 0, st, x, a.ws, gain, a.nvalid, (uint32_t)a.B);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = record(a.events[1], st)) != hipSuccess) return e;
        hipLaunchKernelGGL((wave_pass3_kernel<K, T>), dim3((uint32_t)a.B << Shape<K>::HB),
                           dim3(64), 0, st, a.ws, y, a.nvalid);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        return record(a.events[2], st);
    } else {
        return hipErrorInvalidValue;
    }
}

template <int K, typename T, class Gain>
hipError_t launch_k(const LaunchArgs &a, Gain gain)
{
    if (a.plan == PLAN_TWO_PASS) return launch_two_pass_k<K, T, Gain>(a, gain);
    return a.plan == PLAN_ONE_LAUNCH ? launch_one_launch_k<K, T, Gain>(a, gain)
                                     : launch_wave_tiles_k<K, T, Gain>(a, gain);
}

template <typename T, class Gain>
hipError_t dispatch_k(const LaunchArgs &a, Gain gain)
{
    switch (a.K) {
    case 12: return launch_k<12, T, Gain>(a, gain);
    case 13: return launch_k<13, T, Gain>(a, gain);
    case 14: return launch_k<14, T, Gain>(a, gain);
    case 15: return launch_k<15, T, Gain>(a, gain);
    case 16: return launch_k<16, T, Gain>(a, gain);
    default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t dispatch_gain(const LaunchArgs &a)
{
    if (a.gain_kind == GAIN_LOG_SEPARABLE)
        return dispatch_k<T>(a, tile::LogSeparableGain{a.gain_t, a.gain_c, (uint32_t)a.cbits});
    if (a.B == 1)
        return dispatch_k<T>(a, tile::StreamedGain{a.gain});
    return dispatch_k<T>(a, tile::FullGain{a.gain});
}

}  // namespace wave

hipError_t launch_wave(const LaunchArgs &a)
{
    if (a.plan != PLAN_ONE_LAUNCH && a.plan != PLAN_WAVE_TILES && a.plan != PLAN_TWO_PASS)
        return hipErrorInvalidValue;
    if (a.dtype == DTYPE_BF16)
        return wave::dispatch_gain<__bf16>(a);
    return wave::dispatch_gain<float>(a);
}

}  // namespace whtmix
