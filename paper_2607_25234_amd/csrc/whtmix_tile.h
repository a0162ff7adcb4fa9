// Tile machinery shared by the WHTMix forward and backward kernels (gfx950).
//
// A workgroup owns a tile of 2^M elements (11 <= M <= 15) with tile-local
// index t.  Each of its 2^(M-5) threads holds 32 values in registers.  A
// "layout S" gives thread tau the 32 values whose t has register index k in
// bits [S, S+5) and tau in the remaining bits:
//     t = (tau mod 2^S) | (k << S) | ((tau >> S) << (S + 5)).
// In a layout, a butterfly over t-bit S+j is a register butterfly over bit j
// of k.  The tile's bits are transformed in groups of up to five: the top
// group [M-5, M) straight from the global load (lanes run over the low t
// bits, so loads coalesce), then groups [W, W+5), [W+5, W+10), ... from the
// bottom, each reached by writing the tile to LDS in the old layout and
// reading it back in the new one.  LDS addresses are padded by one word per
// 32 (p = t + t/32), which keeps every layout's reads and writes free of
// bank conflicts and keeps each register's LDS address a constant offset from
// a per-thread base.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "whtmix_plan.h"

namespace whtmix {
namespace tile {

constexpr int VB = 5;        // log2(values per thread)
constexpr int V = 1 << VB;   // values per thread

// ---------------------------------------------------------------- memory
// Global memory is reached through raw buffer resources: a per-tile base and
// byte extent in SGPRs, a 32-bit per-thread offset in one VGPR, and each
// register's constant offset in an SGPR (soffset), so addressing costs no
// 64-bit vector arithmetic and no per-register VGPRs.
constexpr int kRawBufferWord3 = 0x00020000;   // gfx9-family raw buffer descriptor

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes,
                                             kRawBufferWord3);
}

// Cache policy of a buffer access (the instruction's aux bits): temporal for
// the workspace, which is re-read by the next pass and benefits from staying
// in the Infinity Cache; non-temporal (streaming) for x and y, each touched
// once per call, so they do not displace the workspace (measured 2% faster
// per step on the stereo64k workload).
constexpr int kTemporal = 0;
constexpr int kStreaming = 2;   // nt

template <typename T>
struct Elt;

template <>
struct Elt<float> {
    static constexpr uint32_t bytes = 4;
    template <int CP = kTemporal>
    __device__ static __forceinline__ float load(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                 uint32_t soff)
    {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, CP));
    }
    template <int CP = kTemporal>
    __device__ static __forceinline__ void store(float v, __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                 uint32_t soff)
    {
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, voff, soff, CP);
    }
};

template <>
struct Elt<__bf16> {
    static constexpr uint32_t bytes = 2;
    // bf16 -> float32 is exact: the bf16 bits are the high half of the float
    template <int CP = kTemporal>
    __device__ static __forceinline__ float load(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                 uint32_t soff)
    {
        const unsigned short u = __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, CP);
        return __builtin_bit_cast(float, (uint32_t)u << 16);
    }
    // round to nearest even (v_cvt_pk_bf16_f32 on gfx950)
    template <int CP = kTemporal>
    __device__ static __forceinline__ void store(float v, __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                                 uint32_t soff)
    {
        const __bf16 h = (__bf16)v;
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, h), r, voff, soff,
                                              CP);
    }
};

// ---------------------------------------------------------------- layouts
template <int S>
__device__ __forceinline__ uint32_t layout_base(uint32_t tau)
{
    return (tau & ((1u << S) - 1u)) | ((tau >> S) << (S + VB));
}

__host__ __device__ constexpr uint32_t pad(uint32_t t) { return t + (t >> 5); }

// Tile bits [WT, M) are transformed; [0, WT) are carried untouched.
template <int M, int WT>
struct Groups {
    static constexpr int TOP = M - VB;
    // first register bit of the top group that is a transformed tile bit
    static constexpr int JT = WT > TOP ? WT - TOP : 0;
    static constexpr int NBOT = TOP > WT ? (TOP - WT + VB - 1) / VB : 0;
    static constexpr int S(int i) { return WT + VB * i; }
    static constexpr int NB(int i) { return (TOP - S(i)) < VB ? (TOP - S(i)) : VB; }
    static constexpr int SL = NBOT > 0 ? WT + VB * (NBOT - 1) : TOP;
};

// Butterflies over register bits [J0, J1): (a, b) -> (a + b, a - b).
template <int J0, int J1>
__device__ __forceinline__ void butterflies(float (&v)[V])
{
#pragma unroll
    for (int j = J0; j < J1; ++j) {
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

// Re-lay the tile from layout SA to layout SB through LDS.  LEAD: wait first
// for every thread's reads of the previous exchange (not needed the first time
// the tile's LDS is used).
template <int SA, int SB, bool LEAD = true>
__device__ __forceinline__ void exchange(float *lds, float (&v)[V], uint32_t tau)
{
    const uint32_t pa = pad(layout_base<SA>(tau));
    const uint32_t pb = pad(layout_base<SB>(tau));
    if (LEAD)
        __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pa + pad((uint32_t)k << SA)] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        v[k] = lds[pb + pad((uint32_t)k << SB)];
}

// Forward bottom groups I, I+1, ... starting from layout SPREV.  LEAD0:
// wait before the first exchange (needed unless this is the first use of the
// tile's LDS in the kernel).
template <int M, int WT, int I, int SPREV, bool LEAD0 = false>
__device__ __forceinline__ void forward_groups(float *lds, float (&v)[V], uint32_t tau)
{
    using G = Groups<M, WT>;
    if constexpr (I < G::NBOT) {
        constexpr int S = G::S(I);
        exchange<SPREV, S, (I > 0 || LEAD0)>(lds, v, tau);
        butterflies<0, G::NB(I)>(v);
        forward_groups<M, WT, I + 1, S>(lds, v, tau);
    }
}

// Inverse bottom groups I, I-1, ..., 0 (data in group I's layout), ending in
// the top layout.
template <int M, int WT, int I>
__device__ __forceinline__ void inverse_groups(float *lds, float (&v)[V], uint32_t tau)
{
    using G = Groups<M, WT>;
    if constexpr (I >= 0) {
        constexpr int S = G::S(I);
        constexpr int SNEXT = I == 0 ? G::TOP : G::S(I - 1);
        butterflies<0, G::NB(I)>(v);
        exchange<S, SNEXT>(lds, v, tau);
        inverse_groups<M, WT, I - 1>(lds, v, tau);
    }
}

// ---------------------------------------------------------------- vector-first layout
// Outer passes move x and y with 16-byte accesses: 2^VW elements (VW = 3 for
// bf16, 2 for float32) of consecutive t per access.  Their first layout puts
// t bits [0, VW) and [M - 5 + VW, M) in the registers:
//     t = (k mod 2^VW) | (tau << VW) | ((k >> VW) << (M - 5 + VW)),
// so register group j of 2^VW is one access.  The windows then cover
// [VW, M - 5 + VW) from the bottom, as Groups does from bit 0.  Writes from
// this layout to LDS hit 32 distinct banks per half-wave (the pad of one word
// per 32 spreads the 2^VW-strided lanes), like the window layouts.
template <int M, int VWID>
struct VGroups {
    static constexpr int TOPHI = M - VB + VWID;               // first top bit
    static constexpr int NBOT = (M - VB + VB - 1) / VB;
    static constexpr int S(int i) { return VWID + VB * i; }
    static constexpr int NB(int i) { return (TOPHI - S(i)) < VB ? (TOPHI - S(i)) : VB; }
    static constexpr int SL = VWID + VB * (NBOT - 1);
    static_assert(VWID > 0 && SL + VB <= M, "vector-first layout needs a larger tile");
    __device__ static __forceinline__ uint32_t base(uint32_t tau) { return tau << VWID; }
    __host__ __device__ static constexpr uint32_t reg(uint32_t k)
    {
        return (k & ((1u << VWID) - 1u)) | ((k >> VWID) << TOPHI);
    }
};

// Vector width (log2 elements per 16-byte access) the outer passes use for a
// 2^M tile of elements of `bytes` bytes, or 0 for per-element accesses.
// bf16 only: its per-element accesses move 2 bytes per lane, and 16-byte ones
// measured 4-6% faster per step (stereo64k, stereo256k); float32 per-element
// accesses already move 4 bytes per lane and the vector-first layout measured
// no better (within +-4% per kernel on stereo16k and text4k).  The layout
// itself works for float32 (VW = 2, tiles from 2^12).
constexpr int vec_width(int M, int bytes)
{
    const int vw = bytes == 2 ? 3 : 0;
    return vw > 0 && vw + VB * ((M - VB + VB - 1) / VB) <= M ? vw : 0;
}

// From the vector-first layout to window SB (the tile's first use of LDS).
template <int M, int VWID, int SB>
__device__ __forceinline__ void exchange_from_vec(float *lds, float (&v)[V], uint32_t tau)
{
    using VG = VGroups<M, VWID>;
    const uint32_t pa = pad(VG::base(tau));
    const uint32_t pb = pad(layout_base<SB>(tau));
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pa + pad(VG::reg((uint32_t)k))] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        v[k] = lds[pb + pad((uint32_t)k << SB)];
}

// From window SA to the vector-first layout.
template <int M, int VWID, int SA>
__device__ __forceinline__ void exchange_to_vec(float *lds, float (&v)[V], uint32_t tau)
{
    using VG = VGroups<M, VWID>;
    const uint32_t pa = pad(layout_base<SA>(tau));
    const uint32_t pb = pad(VG::base(tau));
    __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pa + pad((uint32_t)k << SA)] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < V; ++k)
        v[k] = lds[pb + pad(VG::reg((uint32_t)k))];
}

// Forward windows I, I+1, ... after the vector-first group (LEAD0: wait for
// earlier readers of the LDS before the first write).
template <int M, int VWID, int I, bool LEAD0 = false>
__device__ __forceinline__ void vforward_groups(float *lds, float (&v)[V], uint32_t tau)
{
    using VG = VGroups<M, VWID>;
    if constexpr (I < VG::NBOT) {
        constexpr int S = VG::S(I);
        if constexpr (I == 0) {
            if (LEAD0)
                __syncthreads();
            exchange_from_vec<M, VWID, S>(lds, v, tau);
        } else {
            exchange<VG::S(I - 1), S>(lds, v, tau);
        }
        butterflies<0, VG::NB(I)>(v);
        vforward_groups<M, VWID, I + 1>(lds, v, tau);
    }
}

// Inverse windows I, I-1, ..., 0 (data in window I's layout), ending in the
// vector-first layout.
template <int M, int VWID, int I>
__device__ __forceinline__ void vinverse_groups(float *lds, float (&v)[V], uint32_t tau)
{
    using VG = VGroups<M, VWID>;
    if constexpr (I >= 0) {
        constexpr int S = VG::S(I);
        butterflies<0, VG::NB(I)>(v);
        if constexpr (I == 0)
            exchange_to_vec<M, VWID, S>(lds, v, tau);
        else
            exchange<S, VG::S(I - 1)>(lds, v, tau);
        vinverse_groups<M, VWID, I - 1>(lds, v, tau);
    }
}

// ---------------------------------------------------------------- address maps
// Each map sends tile-local t to an element offset from the tile's base by
// moving bit fields, so map(a | b) = map(a) + map(b) for disjoint a, b: the
// per-register offsets map(k << S) are compile-time constants.
struct ContigMap {
    __host__ __device__ static constexpr uint32_t at(uint32_t t) { return t; }
};
// Outer-pass chunk index lo (A bits) -> workspace: runs of 2^R elements, run
// number lo >> R strided by a whole middle tile (2^(HB+R)).
template <int HB, int R>
struct RunMap {
    __host__ __device__ static constexpr uint32_t at(uint32_t t)
    {
        return ((t >> R) << (HB + R)) | (t & ((1u << R) - 1u));
    }
};
// Middle tile index (hi << R | run) -> flat slice index hi * 2^A + run.
template <int A, int R>
struct GainMap {
    __host__ __device__ static constexpr uint32_t at(uint32_t t)
    {
        return ((t >> R) << A) | (t & ((1u << R) - 1u));
    }
};

// soff0: a uniform byte offset added to every register's (a second
// register set of a 2^16 tile).
template <int S, class Map, typename T, int CP = kTemporal>
__device__ __forceinline__ void load_layout(float (&v)[V], __amdgpu_buffer_rsrc_t r, uint32_t tau,
                                            uint32_t soff0 = 0)
{
    const uint32_t voff = Map::at(layout_base<S>(tau)) * Elt<T>::bytes;
#pragma unroll
    for (int k = 0; k < V; ++k)
        v[k] = Elt<T>::template load<CP>(r, voff,
                                         soff0 + Map::at((uint32_t)k << S) * Elt<T>::bytes);
}

template <int S, class Map, typename T, int CP = kTemporal>
__device__ __forceinline__ void store_layout(const float (&v)[V], __amdgpu_buffer_rsrc_t r,
                                             uint32_t tau, uint32_t soff0 = 0)
{
    const uint32_t voff = Map::at(layout_base<S>(tau)) * Elt<T>::bytes;
#pragma unroll
    for (int k = 0; k < V; ++k)
        Elt<T>::template store<CP>(v[k], r, voff,
                                   soff0 + Map::at((uint32_t)k << S) * Elt<T>::bytes);
}

// Masked forms for the one tile of a zero-padded slice that straddles the
// last real token: elements with tile index >= valid read as 0 and are not
// stored.  Tiles wholly inside the slice take the unmasked forms; tiles wholly
// in the padding skip their loads.  (The choice is uniform per workgroup.)
template <int S, class Map, typename T>
__device__ __forceinline__ void load_layout_masked(float (&v)[V], __amdgpu_buffer_rsrc_t r,
                                                   uint32_t tau, uint32_t valid)
{
    const uint32_t tb = layout_base<S>(tau);
    const uint32_t voff = Map::at(tb) * Elt<T>::bytes;
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const uint32_t t = tb | ((uint32_t)k << S);
        v[k] = t < valid ? Elt<T>::template load<kStreaming>(
                               r, voff, Map::at((uint32_t)k << S) * Elt<T>::bytes)
                         : 0.0f;
    }
}

template <int S, class Map, typename T>
__device__ __forceinline__ void store_layout_masked(const float (&v)[V],
                                                    __amdgpu_buffer_rsrc_t r, uint32_t tau,
                                                    uint32_t valid)
{
    const uint32_t tb = layout_base<S>(tau);
    const uint32_t voff = Map::at(tb) * Elt<T>::bytes;
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const uint32_t t = tb | ((uint32_t)k << S);
        if (t < valid)
            Elt<T>::template store<kStreaming>(v[k], r, voff,
                                               Map::at((uint32_t)k << S) * Elt<T>::bytes);
    }
}

// A contiguous tile of 2^M elements of x (type T) with `valid` real elements
// (streaming cache policy).
template <int S, int M, typename T>
__device__ __forceinline__ void load_tile(float (&v)[V], const T *base, uint32_t valid,
                                          uint32_t tau)
{
    if (valid >= (1u << M)) {
        load_layout<S, ContigMap, T, kStreaming>(v, buffer(base, (1u << M) * Elt<T>::bytes), tau);
    } else if (valid == 0) {
#pragma unroll
        for (int k = 0; k < V; ++k)
            v[k] = 0.0f;
    } else {
        load_layout_masked<S, ContigMap, T>(v, buffer(base, valid * Elt<T>::bytes), tau, valid);
    }
}

template <int S, int M, typename T>
__device__ __forceinline__ void store_tile(const float (&v)[V], T *base, uint32_t valid,
                                           uint32_t tau)
{
    if (valid >= (1u << M))
        store_layout<S, ContigMap, T, kStreaming>(v, buffer(base, (1u << M) * Elt<T>::bytes),
                                                  tau);
    else if (valid > 0)
        store_layout_masked<S, ContigMap, T>(v, buffer(base, valid * Elt<T>::bytes), tau, valid);
}

typedef unsigned int vu32x4 __attribute__((ext_vector_type(4)));
typedef float vf32x4 __attribute__((ext_vector_type(4)));

// A tile of 2^M elements in the vector-first layout, 16-byte accesses
// (streaming cache policy).  Partial tiles (the straddling tile of a padded
// slice) take per-element masked accesses in the same layout.  Whole vectors
// are bit-cast and then indexed: a bit_cast of one ext-vector element reads
// element 0 in this toolchain.
template <int M, int VWID, typename T>
__device__ __forceinline__ void load_tile_vec(float (&v)[V], const T *base, uint32_t valid,
                                              uint32_t tau)
{
    using VG = VGroups<M, VWID>;
    constexpr int PER = 1 << VWID;   // elements per access
    static_assert(PER * (int)sizeof(T) == 16, "16-byte accesses");
    if (valid >= (1u << M)) {
        const __amdgpu_buffer_rsrc_t r = buffer(base, (1u << M) * Elt<T>::bytes);
        const uint32_t voff = VG::base(tau) * Elt<T>::bytes;
#pragma unroll
        for (int j = 0; j < V / PER; ++j) {
            const vu32x4 q = __builtin_bit_cast(
                vu32x4, __builtin_amdgcn_raw_buffer_load_b128(
                            r, voff, VG::reg((uint32_t)(j * PER)) * Elt<T>::bytes, kStreaming));
            if constexpr (sizeof(T) == 4) {
                const vf32x4 f = __builtin_bit_cast(vf32x4, q);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[j * PER + e] = f[e];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t w = q[e];
                    v[j * PER + 2 * e] = __builtin_bit_cast(float, w << 16);
                    v[j * PER + 2 * e + 1] = __builtin_bit_cast(float, w & 0xffff0000u);
                }
            }
        }
    } else if (valid == 0) {
#pragma unroll
        for (int k = 0; k < V; ++k)
            v[k] = 0.0f;
    } else {
        const __amdgpu_buffer_rsrc_t r = buffer(base, valid * Elt<T>::bytes);
        const uint32_t tb = VG::base(tau);
#pragma unroll
        for (int k = 0; k < V; ++k) {
            const uint32_t t = tb | VG::reg((uint32_t)k);
            v[k] = t < valid ? Elt<T>::template load<kStreaming>(r, tb * Elt<T>::bytes,
                                                                 VG::reg((uint32_t)k) *
                                                                     Elt<T>::bytes)
                             : 0.0f;
        }
    }
}

template <int M, int VWID, typename T>
__device__ __forceinline__ void store_tile_vec(const float (&v)[V], T *base, uint32_t valid,
                                               uint32_t tau)
{
    using VG = VGroups<M, VWID>;
    constexpr int PER = 1 << VWID;
    static_assert(PER * (int)sizeof(T) == 16, "16-byte accesses");
    if (valid >= (1u << M)) {
        const __amdgpu_buffer_rsrc_t r = buffer(base, (1u << M) * Elt<T>::bytes);
        const uint32_t voff = VG::base(tau) * Elt<T>::bytes;
#pragma unroll
        for (int j = 0; j < V / PER; ++j) {
            vu32x4 q;
            if constexpr (sizeof(T) == 4) {
                const vf32x4 f = {v[j * PER], v[j * PER + 1], v[j * PER + 2], v[j * PER + 3]};
                q = __builtin_bit_cast(vu32x4, f);
            } else {   // round to nearest even, two bf16 per word
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t lo =
                        __builtin_bit_cast(unsigned short, (__bf16)v[j * PER + 2 * e]);
                    const uint32_t hi =
                        __builtin_bit_cast(unsigned short, (__bf16)v[j * PER + 2 * e + 1]);
                    q[e] = lo | (hi << 16);
                }
            }
            __builtin_amdgcn_raw_buffer_store_b128(q, r, voff,
                                                   VG::reg((uint32_t)(j * PER)) * Elt<T>::bytes,
                                                   kStreaming);
        }
    } else if (valid > 0) {
        const __amdgpu_buffer_rsrc_t r = buffer(base, valid * Elt<T>::bytes);
        const uint32_t tb = VG::base(tau);
#pragma unroll
        for (int k = 0; k < V; ++k) {
            const uint32_t t = tb | VG::reg((uint32_t)k);
            if (t < valid)
                Elt<T>::template store<kStreaming>(v[k], r, tb * Elt<T>::bytes,
                                                   VG::reg((uint32_t)k) * Elt<T>::bytes);
        }
    }
}

// ---------------------------------------------------------------- gains
// f is the flat index n*C + c of the (padded) slice.  The gain is read with
// plain global loads: for its 128-byte-run pattern they measured markedly
// faster than buffer loads on gfx950.  It is requested right after the data
// tile so its latency overlaps the forward butterflies.

// Joint per-frequency gain G[N_pad][C] (linear).  NT: the middle pass's
// loads (MIDDLE) are non-temporal.  The host picks it for a batch of one
// slice, whose middle pass reads each gain element exactly once, so the gain
// does not displace the workspace in the Infinity Cache (stereo256k 334 ->
// 309 us per step), and for gains of 16 MiB and more (with_forward_middle_gain).
// With more slices each gain tile is read once per slice on one XCD, and for
// small gains temporal loads let those reads hit (non-temporal ones cost
// text4k, 32 slices, 38 -> 42 us).  A type, not a run-time flag: the
// compiler merges the loads of the two branches of a flag and drops the hint.
template <bool NT>
struct FullGainT {
    const float *g;
    // Each register's base (uniform) is a scalar pointer into global memory
    // and the thread's part a 32-bit byte offset, so every load is one
    // global_load with a scalar base: no 64-bit vector address per register,
    // and (unlike a flat load) no share of the LDS wait counter.
    template <int S, class Map, bool MIDDLE = false>
    __device__ __forceinline__ void load(float (&gv)[V], uint32_t f0, uint32_t tau) const
    {
        typedef const __attribute__((address_space(1))) float gfloat;
        const uint32_t voff = Map::at(layout_base<S>(tau)) * 4u;
#pragma unroll
        for (int k = 0; k < V; ++k) {
            const char *row = reinterpret_cast<const char *>(g + f0 + Map::at((uint32_t)k << S));
            asm("" : "+s"(row));   // opaque scalar base: not re-associated into a vector one
            gfloat *p = (gfloat *)(row + voff);
            if constexpr (NT && MIDDLE)
                gv[k] = __builtin_nontemporal_load(p);
            else
                gv[k] = *p;
        }
    }
    __device__ __forceinline__ float at(uint32_t f) const { return g[f]; }
};
using FullGain = FullGainT<false>;
using StreamedGain = FullGainT<true>;

// Calls f with the gain a middle pass over `slices` slices reads: the
// streamed form of a joint gain for one slice, else the gain itself.
template <class Gain, class F>
inline hipError_t with_middle_gain(Gain gain, int64_t, F &&f)
{
    return f(gain);
}
template <class F>
inline hipError_t with_middle_gain(FullGain gain, int64_t slices, F &&f)
{
    return slices == 1 ? f(StreamedGain{gain.g}) : f(gain);
}

// The forward middle pass also streams a joint gain of 2^22 elements (16 MiB)
// or more whatever the batch: keeping the workspace in the Infinity Cache
// then outweighs the L2 hits of the slices that share a gain tile
// (stereo64k, four slices of 2^23: 120.6 -> 118.5 us per step).  Smaller
// gains keep temporal loads (stereo16k and text4k measured slower streamed).
constexpr int kStreamGainMinK = 22;
template <class Gain, class F>
inline hipError_t with_forward_middle_gain(Gain gain, int64_t slices, int, F &&f)
{
    return with_middle_gain(gain, slices, f);
}
template <class F>
inline hipError_t with_forward_middle_gain(FullGain gain, int64_t slices, int K, F &&f)
{
    return slices == 1 || K >= kStreamGainMinK ? f(StreamedGain{gain.g}) : f(gain);
}

// The paper's parametrisation (eqs. (2)-(3)): log-domain gains g_t[N_pad]
// over token frequencies and g_c[C] over channel frequencies; the gain of
// frequency (n, c) is exp(g_t[n]) * exp(g_c[c]), computed as one exp of the
// sum.
struct LogSeparableGain {
    const float *gt;
    const float *gc;
    uint32_t cbits;   // log2(C)
    // exp via the hardware exp2 (v_exp_f32) of x*log2(e): relative error
    // about 1e-7 for log gains of moderate size, far inside the tolerances.
    __device__ __forceinline__ float at(uint32_t f) const
    {
        return __expf(gt[f >> cbits] + gc[f & ((1u << cbits) - 1u)]);
    }
    template <int S, class Map, bool MIDDLE = false>
    __device__ __forceinline__ void load(float (&gv)[V], uint32_t f0, uint32_t tau) const
    {
        const uint32_t fb = f0 + Map::at(layout_base<S>(tau));
#pragma unroll
        for (int k = 0; k < V; ++k)
            gv[k] = at(fb + Map::at((uint32_t)k << S));
    }
};

// v *= gain * 2^-K (gain already gathered in the same layout).
template <int K>
__device__ __forceinline__ void apply_gain(float (&v)[V], const float (&g)[V])
{
    constexpr float scale = 1.0f / (float)(1u << K);   // exact power of two
#pragma unroll
    for (int k = 0; k < V; ++k)
        v[k] *= g[k] * scale;
}

// Byte extent of a map over a tile of 2^M elements (largest offset + 1).
template <class Map, int M, typename T>
constexpr uint32_t extent_bytes()
{
    return (Map::at((1u << M) - 1u) + 1u) * Elt<T>::bytes;
}


// Outer-pass block renumbering.  With runs shorter than 32 floats (R < 5) a
// 128-byte line of the workspace holds the runs of 2^(5-R) neighbouring hi
// blocks.  Blocks are dealt round-robin over the 8 XCDs (block i on XCD
// i mod 8), so blocks i, i+8, i+16, ... share an XCD and its L2: they are
// given consecutive hi, and each line is then filled (or read) by one XCD.
// The map is a permutation within groups of 8 * 2^(5-R) blocks; grids that
// are not a multiple of the group keep the identity.
template <int R>
__device__ __forceinline__ uint32_t outer_block(uint32_t blk, uint32_t nblk)
{
    if constexpr (R >= 5) {
        return blk;
    } else {
        constexpr uint32_t g = 1u << (5 - R);
        if (nblk % (8u * g) != 0)
            return blk;
        return (blk & ~(8u * g - 1u)) | ((blk & 7u) * g) | ((blk >> 3) & (g - 1u));
    }
}

// Number of real elements in the outer tile hi of a zero-padded slice.
template <int A>
__device__ __forceinline__ uint32_t tile_valid(uint32_t nvalid, uint32_t hi)
{
    const uint32_t start = hi << A;
    return nvalid <= start ? 0u : min(nvalid - start, 1u << A);
}

// OUTER_FWD tile (forward pass and backward pass): block = b * 2^HB + hi;
// the chunk x[b][hi * 2^A ...] (nvalid real elements per slice, the rest
// zero padding) is transformed over its A bits and stored to the workspace
// in runs of 2^R, so that each middle tile is contiguous.
// VWID > 0: x is read with 16-byte accesses in the vector-first layout (the
// launcher checks that every slice starts 16-byte aligned).
template <int A, int HB, int R, typename T, int VWID>
__device__ __forceinline__ void outer_fwd_tile(float *lds, const T *__restrict__ x,
                                               float *__restrict__ ws, uint32_t nvalid,
                                               uint32_t blk)
{
    using Run = RunMap<HB, R>;
    const uint32_t tau = threadIdx.x;
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const T *src = x + b * nvalid + ((size_t)hi << A);
    const __amdgpu_buffer_rsrc_t r =
        buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>());
    float v[V];
    if constexpr (VWID > 0) {
        using VG = VGroups<A, VWID>;
        load_tile_vec<A, VWID, T>(v, src, tile_valid<A>(nvalid, hi), tau);
        butterflies<0, VB>(v);
        vforward_groups<A, VWID, 0>(lds, v, tau);
        store_layout<VG::SL, Run, float>(v, r, tau);
    } else {
        using G = Groups<A, 0>;
        load_tile<G::TOP, A, T>(v, src, tile_valid<A>(nvalid, hi), tau);
        butterflies<0, VB>(v);
        forward_groups<A, 0, 0, G::TOP>(lds, v, tau);
        store_layout<G::SL, Run, float>(v, r, tau);
    }
}

template <int A, int HB, int R, typename T, int VWID>
__global__ void __launch_bounds__(1 << (A - VB))
outer_fwd_kernel(const T *__restrict__ x, float *__restrict__ ws, uint32_t nvalid)
{
    __shared__ float lds[pad(1u << A)];
    outer_fwd_tile<A, HB, R, T, VWID>(lds, x, ws, nvalid, outer_block<R>(blockIdx.x, gridDim.x));
}

// OUTER_FWD of two operands in one launch (the backward pass's x and dy):
// the first half of the grid takes x into wsx, the second dy into wsd.  Each
// half is numbered as a grid of its own; the halves start on the same XCD
// whenever the renumbering of outer_block applies (it needs a half that is a
// multiple of 8 blocks).
template <int A, int HB, int R, typename T, int VWID>
__global__ void __launch_bounds__(1 << (A - VB))
outer_fwd2_kernel(const T *__restrict__ x, const T *__restrict__ dy, float *__restrict__ wsx,
                  float *__restrict__ wsd, uint32_t nvalid)
{
    __shared__ float lds[pad(1u << A)];
    const uint32_t half = gridDim.x >> 1;
    const bool second = blockIdx.x >= half;
    const uint32_t blk = outer_block<R>(blockIdx.x - (second ? half : 0u), half);
    outer_fwd_tile<A, HB, R, T, VWID>(lds, second ? dy : x, second ? wsd : wsx, nvalid, blk);
}

// OUTER_INV kernel: the mirror of OUTER_FWD (inverse over the A low bits of
// each workspace chunk, then the store of y).
template <int A, int HB, int R, typename T, int VWID>
__global__ void __launch_bounds__(1 << (A - VB))
outer_inv_kernel(const float *__restrict__ ws, T *__restrict__ y, uint32_t nvalid)
{
    using Run = RunMap<HB, R>;
    __shared__ float lds[pad(1u << A)];
    const uint32_t tau = threadIdx.x;
    const uint32_t blk = outer_block<R>(blockIdx.x, gridDim.x);
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const uint32_t valid = tile_valid<A>(nvalid, hi);
    if (valid == 0)
        return;   // wholly padding: nothing to store (uniform per workgroup)
    const __amdgpu_buffer_rsrc_t r =
        buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>());
    T *dst = y + b * nvalid + ((size_t)hi << A);
    float v[V];
    if constexpr (VWID > 0) {
        using VG = VGroups<A, VWID>;
        load_layout<VG::SL, Run, float>(v, r, tau);
        vinverse_groups<A, VWID, VG::NBOT - 1>(lds, v, tau);
        butterflies<0, VB>(v);
        store_tile_vec<A, VWID, T>(v, dst, valid, tau);
    } else {
        using G = Groups<A, 0>;
        load_layout<G::SL, Run, float>(v, r, tau);
        inverse_groups<A, 0, G::NBOT - 1>(lds, v, tau);
        butterflies<0, VB>(v);
        store_tile<G::TOP, A, T>(v, dst, valid, tau);
    }
}

// ---------------------------------------------------------------- 2^16 outer tiles
// Slices of 2^26 elements and more use outer tiles of 2^16 (three_pass_split):
// a workgroup of 1024 threads holds two 2^15 sub-tiles (tile bit 15 = 0 and
// 1) in two register sets.  Bit 15 is a butterfly between the sets; bits
// 0..14 are the 2^15 schedule above, run on each set in turn through the
// same LDS.  The RunMap offsets are additive, so the second set's workspace
// offsets are the first's plus RunMap(2^15).

// (a, b) -> (a + b, a - b) between the two register sets.
__device__ __forceinline__ void cross_butterflies(float (&v0)[V], float (&v1)[V])
{
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const float a = v0[k], b = v1[k];
        v0[k] = a + b;
        v1[k] = a - b;
    }
}

template <int HB, int R, typename T, int VWID>
__device__ __forceinline__ void outer_fwd_tile2(float *lds, const T *__restrict__ x,
                                                float *__restrict__ ws, uint32_t nvalid,
                                                uint32_t blk)
{
    constexpr int A = 16, M = 15;
    using Run = RunMap<HB, R>;
    const uint32_t tau = threadIdx.x;
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const uint32_t valid = tile_valid<A>(nvalid, hi);
    const uint32_t valid0 = min(valid, 1u << M);
    const uint32_t valid1 = valid > (1u << M) ? valid - (1u << M) : 0u;
    const T *base = x + b * nvalid + ((size_t)hi << A);
    const __amdgpu_buffer_rsrc_t r =
        buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>());
    float v0[V], v1[V];
    if constexpr (VWID > 0) {
        using VG = VGroups<M, VWID>;
        load_tile_vec<M, VWID, T>(v0, base, valid0, tau);
        load_tile_vec<M, VWID, T>(v1, base + (1u << M), valid1, tau);
        cross_butterflies(v0, v1);
        butterflies<0, VB>(v0);
        butterflies<0, VB>(v1);
        vforward_groups<M, VWID, 0>(lds, v0, tau);
        store_layout<VG::SL, Run, float>(v0, r, tau);   // in flight through set 1's exchanges
        vforward_groups<M, VWID, 0, true>(lds, v1, tau);
        store_layout<VG::SL, Run, float>(v1, r, tau, Run::at(1u << M) * 4u);
    } else {
        using G = Groups<M, 0>;
        load_tile<G::TOP, M, T>(v0, base, valid0, tau);
        load_tile<G::TOP, M, T>(v1, base + (1u << M), valid1, tau);
        cross_butterflies(v0, v1);
        butterflies<0, VB>(v0);
        butterflies<0, VB>(v1);
        forward_groups<M, 0, 0, G::TOP>(lds, v0, tau);
        store_layout<G::SL, Run, float>(v0, r, tau);
        forward_groups<M, 0, 0, G::TOP, true>(lds, v1, tau);
        store_layout<G::SL, Run, float>(v1, r, tau, Run::at(1u << M) * 4u);
    }
}

template <int HB, int R, typename T, int VWID>
__global__ void __launch_bounds__(1 << (15 - VB))
outer_fwd_kernel2(const T *__restrict__ x, float *__restrict__ ws, uint32_t nvalid)
{
    __shared__ float lds[pad(1u << 15)];
    outer_fwd_tile2<HB, R, T, VWID>(lds, x, ws, nvalid, outer_block<R>(blockIdx.x, gridDim.x));
}

// OUTER_FWD over 2^16 tiles, bf16 x in 16-byte groups, as a grid of one
// resident workgroup per CU that takes tiles blockIdx.x, blockIdx.x +
// gridDim.x, ...: the next tile's x (both register sets, 32 words per
// thread, when the tile is whole) is loaded while this tile is transformed
// and stored, since one 1024-thread workgroup per CU leaves no other
// workgroup to cover the load latency.  With two operands (x1, ws1 not
// null) tiles ntiles.. 2 ntiles - 1 are those of x1, as in outer_fwd2_kernel2.
template <int HB, int R>
__global__ void __launch_bounds__(1 << (15 - VB))
outer_fwd_kernel2_pf(const __bf16 *__restrict__ x0, float *__restrict__ ws0,
                     const __bf16 *__restrict__ x1, float *__restrict__ ws1, uint32_t nvalid,
                     uint32_t ntiles)
{
    constexpr int A = 16, M = 15, VWID = 3, PER = 8, NQ = V / PER;
    using VG = VGroups<M, VWID>;
    using Run = RunMap<HB, R>;
    __shared__ float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t voff = VG::base(tau) * 2u;
    vu32x4 raw[2][NQ];
    const uint32_t total = x1 ? 2u * ntiles : ntiles;
    // operand and tile of grid-wide tile t
    auto locate = [&](uint32_t t, bool &second) -> uint32_t {
        second = t >= ntiles;
        return outer_block<R>(second ? t - ntiles : t, ntiles);
    };
    // issue the loads of grid-wide tile t into raw; false (nothing issued)
    // for a partial tile, which the loop loads itself
    auto issue = [&](uint32_t t) -> bool {
        bool second;
        const uint32_t blk = locate(t, second);
        const uint32_t hi = blk & ((1u << HB) - 1u);
        if (tile_valid<A>(nvalid, hi) < (1u << A))
            return false;   // uniform per workgroup
        const __bf16 *base =
            (second ? x1 : x0) + (size_t)(blk >> HB) * nvalid + ((size_t)hi << A);
        const __amdgpu_buffer_rsrc_t r0 = buffer(base, (1u << M) * 2u);
        const __amdgpu_buffer_rsrc_t r1 = buffer(base + (1u << M), (1u << M) * 2u);
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
            raw[0][j] = __builtin_bit_cast(
                vu32x4, __builtin_amdgcn_raw_buffer_load_b128(
                            r0, voff, VG::reg((uint32_t)(j * PER)) * 2u, kStreaming));
            raw[1][j] = __builtin_bit_cast(
                vu32x4, __builtin_amdgcn_raw_buffer_load_b128(
                            r1, voff, VG::reg((uint32_t)(j * PER)) * 2u, kStreaming));
        }
        return true;
    };
    // tile t is worked on XCD t mod 8, as in the one-tile-per-workgroup grid
    // (the grid is a multiple of 8 or covers every tile), so outer_block's
    // renumbering applies unchanged
    uint32_t t = blockIdx.x;
    bool have = t < total && issue(t);
    for (; t < total; t += gridDim.x) {   // uniform per workgroup
        bool second;
        const uint32_t blk = locate(t, second);
        const uint32_t hi = blk & ((1u << HB) - 1u);
        const __bf16 *x = second ? x1 : x0;
        float *ws = second ? ws1 : ws0;
        float v0[V], v1[V];
        if (have) {
#pragma unroll
            for (int j = 0; j < NQ; ++j) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t w0 = raw[0][j][e], w1 = raw[1][j][e];
                    v0[j * PER + 2 * e] = __builtin_bit_cast(float, w0 << 16);
                    v0[j * PER + 2 * e + 1] = __builtin_bit_cast(float, w0 & 0xffff0000u);
                    v1[j * PER + 2 * e] = __builtin_bit_cast(float, w1 << 16);
                    v1[j * PER + 2 * e + 1] = __builtin_bit_cast(float, w1 & 0xffff0000u);
                }
            }
        } else {
            const uint32_t valid = tile_valid<A>(nvalid, hi);
            const __bf16 *base = x + (size_t)(blk >> HB) * nvalid + ((size_t)hi << A);
            load_tile_vec<M, VWID, __bf16>(v0, base, min(valid, 1u << M), tau);
            load_tile_vec<M, VWID, __bf16>(v1, base + (1u << M),
                                           valid > (1u << M) ? valid - (1u << M) : 0u, tau);
        }
        have = t + gridDim.x < total && issue(t + gridDim.x);
        const __amdgpu_buffer_rsrc_t r =
            buffer(ws + ((size_t)(blk >> HB) << (A + HB)) + ((size_t)hi << R),
                   extent_bytes<Run, A, float>());
        cross_butterflies(v0, v1);
        butterflies<0, VB>(v0);
        butterflies<0, VB>(v1);
        vforward_groups<M, VWID, 0, true>(lds, v0, tau);
        store_layout<VG::SL, Run, float>(v0, r, tau);
        vforward_groups<M, VWID, 0, true>(lds, v1, tau);
        store_layout<VG::SL, Run, float>(v1, r, tau, Run::at(1u << M) * 4u);
    }
}

// Two operands in one launch (as outer_fwd2_kernel).
template <int HB, int R, typename T, int VWID>
__global__ void __launch_bounds__(1 << (15 - VB))
outer_fwd2_kernel2(const T *__restrict__ x, const T *__restrict__ dy, float *__restrict__ wsx,
                   float *__restrict__ wsd, uint32_t nvalid)
{
    __shared__ float lds[pad(1u << 15)];
    const uint32_t half = gridDim.x >> 1;
    const bool second = blockIdx.x >= half;
    const uint32_t blk = outer_block<R>(blockIdx.x - (second ? half : 0u), half);
    outer_fwd_tile2<HB, R, T, VWID>(lds, second ? dy : x, second ? wsd : wsx, nvalid, blk);
}

template <int HB, int R, typename T, int VWID>
__global__ void __launch_bounds__(1 << (15 - VB))
outer_inv_kernel2(const float *__restrict__ ws, T *__restrict__ y, uint32_t nvalid)
{
    constexpr int A = 16, M = 15;
    using Run = RunMap<HB, R>;
    __shared__ float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t blk = outer_block<R>(blockIdx.x, gridDim.x);
    const size_t b = blk >> HB;
    const uint32_t hi = blk & ((1u << HB) - 1u);
    const uint32_t valid = tile_valid<A>(nvalid, hi);
    if (valid == 0)
        return;   // wholly padding: nothing to store (uniform per workgroup)
    const __amdgpu_buffer_rsrc_t r =
        buffer(ws + (b << (A + HB)) + ((size_t)hi << R), extent_bytes<Run, A, float>());
    T *base = y + b * nvalid + ((size_t)hi << A);
    float v0[V], v1[V];
    if constexpr (VWID > 0) {
        using VG = VGroups<M, VWID>;
        load_layout<VG::SL, Run, float>(v0, r, tau);
        load_layout<VG::SL, Run, float>(v1, r, tau, Run::at(1u << M) * 4u);
        vinverse_groups<M, VWID, VG::NBOT - 1>(lds, v0, tau);
        vinverse_groups<M, VWID, VG::NBOT - 1>(lds, v1, tau);
        butterflies<0, VB>(v0);
        butterflies<0, VB>(v1);
        cross_butterflies(v0, v1);
        store_tile_vec<M, VWID, T>(v0, base, min(valid, 1u << M), tau);
        if (valid > (1u << M))
            store_tile_vec<M, VWID, T>(v1, base + (1u << M), valid - (1u << M), tau);
    } else {
        using G = Groups<M, 0>;
        load_layout<G::SL, Run, float>(v0, r, tau);
        load_layout<G::SL, Run, float>(v1, r, tau, Run::at(1u << M) * 4u);
        inverse_groups<M, 0, G::NBOT - 1>(lds, v0, tau);
        inverse_groups<M, 0, G::NBOT - 1>(lds, v1, tau);
        butterflies<0, VB>(v0);
        butterflies<0, VB>(v1);
        cross_butterflies(v0, v1);
        store_tile<G::TOP, M, T>(v0, base, min(valid, 1u << M), tau);
        if (valid > (1u << M))
            store_tile<G::TOP, M, T>(v1, base + (1u << M), valid - (1u << M), tau);
    }
}

// Launch helpers for the mixer's outer passes (2^11..2^16 tiles).  x and y
// move with 16-byte accesses when the tile allows (vec_width) and every
// slice starts 16-byte aligned (x and y themselves are 16-byte aligned).
template <int A, typename T>
constexpr int outer_vec_width()
{
    return vec_width(A < 15 ? A : 15, (int)sizeof(T));
}

template <int A, typename T>
inline bool use_vec(uint32_t nvalid)
{
    return outer_vec_width<A, T>() > 0 && ((uint64_t)nvalid * sizeof(T)) % 16u == 0;
}

template <int K, typename T>
hipError_t launch_outer_fwd(const T *x, float *ws, int64_t B, uint32_t nvalid, hipStream_t st)
{
    constexpr Split sp = three_pass_split(K);
    constexpr int VW = outer_vec_width<sp.A, T>();
    const dim3 grid((uint32_t)(B << sp.HB));
    const bool vec = use_vec<sp.A, T>(nvalid);
    if constexpr (sp.A == 16) {
        const dim3 block(1u << (15 - VB));
        if constexpr (sizeof(T) == 2 && VW == 3) {
            if (vec) {
                const uint32_t ntiles = (uint32_t)(B << sp.HB);
                hipLaunchKernelGGL((outer_fwd_kernel2_pf<sp.HB, sp.R>),
                                   dim3(ntiles < 256u ? ntiles : 256u), block, 0, st, x, ws,
                                   (const __bf16 *)nullptr, (float *)nullptr, nvalid, ntiles);
                return hipGetLastError();
            }
        }
        if (vec)
            hipLaunchKernelGGL((outer_fwd_kernel2<sp.HB, sp.R, T, VW>), grid, block, 0, st, x, ws,
                               nvalid);
        else
            hipLaunchKernelGGL((outer_fwd_kernel2<sp.HB, sp.R, T, 0>), grid, block, 0, st, x, ws,
                               nvalid);
    } else {
        const dim3 block(1u << (sp.A - VB));
        if (vec)
            hipLaunchKernelGGL((outer_fwd_kernel<sp.A, sp.HB, sp.R, T, VW>), grid, block, 0, st, x,
                               ws, nvalid);
        else
            hipLaunchKernelGGL((outer_fwd_kernel<sp.A, sp.HB, sp.R, T, 0>), grid, block, 0, st, x,
                               ws, nvalid);
    }
    return hipGetLastError();
}

template <int K, typename T>
hipError_t launch_outer_fwd2(const T *x, const T *dy, float *wsx, float *wsd, int64_t B,
                             uint32_t nvalid, hipStream_t st)
{
    constexpr Split sp = three_pass_split(K);
    constexpr int VW = outer_vec_width<sp.A, T>();
    const dim3 grid((uint32_t)(2 * (B << sp.HB)));
    const bool vec = use_vec<sp.A, T>(nvalid);
    if constexpr (sp.A == 16) {
        const dim3 block(1u << (15 - VB));
        if constexpr (sizeof(T) == 2 && VW == 3) {
            if (vec) {
                const uint32_t ntiles = (uint32_t)(B << sp.HB);
                hipLaunchKernelGGL((outer_fwd_kernel2_pf<sp.HB, sp.R>),
                                   dim3(2u * ntiles < 256u ? 2u * ntiles : 256u), block, 0, st, x,
                                   wsx, dy, wsd, nvalid, ntiles);
                return hipGetLastError();
            }
        }
        if (vec)
            hipLaunchKernelGGL((outer_fwd2_kernel2<sp.HB, sp.R, T, VW>), grid, block, 0, st, x, dy,
                               wsx, wsd, nvalid);
        else
            hipLaunchKernelGGL((outer_fwd2_kernel2<sp.HB, sp.R, T, 0>), grid, block, 0, st, x, dy,
                               wsx, wsd, nvalid);
    } else {
        const dim3 block(1u << (sp.A - VB));
        if (vec)
            hipLaunchKernelGGL((outer_fwd2_kernel<sp.A, sp.HB, sp.R, T, VW>), grid, block, 0, st,
                               x, dy, wsx, wsd, nvalid);
        else
            hipLaunchKernelGGL((outer_fwd2_kernel<sp.A, sp.HB, sp.R, T, 0>), grid, block, 0, st, x,
                               dy, wsx, wsd, nvalid);
    }
    return hipGetLastError();
}

template <int K, typename T>
hipError_t launch_outer_inv(const float *ws, T *y, int64_t B, uint32_t nvalid, hipStream_t st)
{
    constexpr Split sp = three_pass_split(K);
    constexpr int VW = outer_vec_width<sp.A, T>();
    const dim3 grid((uint32_t)(B << sp.HB));
    const bool vec = use_vec<sp.A, T>(nvalid);
    if constexpr (sp.A == 16) {
        const dim3 block(1u << (15 - VB));
        if (vec)
            hipLaunchKernelGGL((outer_inv_kernel2<sp.HB, sp.R, T, VW>), grid, block, 0, st, ws, y,
                               nvalid);
        else
            hipLaunchKernelGGL((outer_inv_kernel2<sp.HB, sp.R, T, 0>), grid, block, 0, st, ws, y,
                               nvalid);
    } else {
        const dim3 block(1u << (sp.A - VB));
        if (vec)
            hipLaunchKernelGGL((outer_inv_kernel<sp.A, sp.HB, sp.R, T, VW>), grid, block, 0, st, ws,
                               y, nvalid);
        else
            hipLaunchKernelGGL((outer_inv_kernel<sp.A, sp.HB, sp.R, T, 0>), grid, block, 0, st, ws,
                               y, nvalid);
    }
    return hipGetLastError();
}

}  // namespace tile
}  // namespace whtmix
