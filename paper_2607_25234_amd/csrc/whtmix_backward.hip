// WHTMix backward kernels for gfx950 (MI355X).
//
// The paper trains the mixer's gains (section IV-A).  For a loss with upstream
// gradient dY, on the zero-padded flat slice of L = 2^K elements with the
// orthonormal transform T = L^-1/2 H_L:
//     dX = the mixer applied to dY        (self-adjoint: H symmetric, G
//                                          diagonal) -- the forward kernels;
//     dG = sum over b of T(x_b) o T(dy_b) (in the transform domain).
// dG needs forward-only transforms of x and dy and a product summed over the
// batch.  The batch is split into chunks; each workgroup accumulates its
// chunk in registers and a fixed-order pass adds the chunks, so results do not
// depend on scheduling (no atomics).
//
// For the separable log gains G[n][c] = exp(g_t[n] + g_c[c]):
//     dg_t[n] = sum over c of dG[n][c] G[n][c],  dg_c[c] = sum over n of the same.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "whtmix_launch.h"
#include "whtmix_plan.h"
#include "whtmix_tile.h"

namespace whtmix {
namespace {

using namespace tile;

// Three-pass dG.  After OUTER_FWD of x and of dy over the A low bits, one
// workgroup owns one workspace run (2^HB x 2^R elements) for a chunk of
// slices: forward over the HB high bits for both operands, multiply,
// accumulate; then 2^-K times the sum is stored at the run's positions of G.
template <int A, int HB, int R>
__global__ void __launch_bounds__(1 << (HB + R - VB))
grad_middle_kernel(const float *__restrict__ wsx, const float *__restrict__ wsd,
                   float *__restrict__ out, uint32_t nslices, uint32_t per_chunk)
{
    constexpr int M = HB + R;
    using G = Groups<M, R>;
    using Gain = GainMap<A, R>;
    __shared__ float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t run = blockIdx.x & ((1u << (A - R)) - 1u);
    const uint32_t chunk = blockIdx.x >> (A - R);
    const uint32_t b0 = chunk * per_chunk;
    const uint32_t b1 = min(b0 + per_chunk, nslices);
    float acc[V];
#pragma unroll
    for (int k = 0; k < V; ++k)
        acc[k] = 0.0f;
    for (uint32_t b = b0; b < b1; ++b) {   // uniform over the workgroup
        const size_t off = ((size_t)b << (A + HB)) + ((size_t)run << M);
        float vx[V], vd[V];
        load_layout<G::TOP, ContigMap, float>(vx, buffer(wsx + off, (1u << M) * 4u), tau);
        load_layout<G::TOP, ContigMap, float>(vd, buffer(wsd + off, (1u << M) * 4u), tau);
        butterflies<G::JT, VB>(vx);
        butterflies<G::JT, VB>(vd);
        forward_groups<M, R, 0, G::TOP, true>(lds, vx, tau);
        forward_groups<M, R, 0, G::TOP, true>(lds, vd, tau);
#pragma unroll
        for (int k = 0; k < V; ++k)
            acc[k] = fmaf(vx[k], vd[k], acc[k]);
    }
    constexpr float scale = 1.0f / (float)(1u << (A + HB));
    float *o = out + ((size_t)chunk << (A + HB)) + ((size_t)run << R) +
               Gain::at(layout_base<G::SL>(tau));
#pragma unroll
    for (int k = 0; k < V; ++k)
        o[Gain::at((uint32_t)k << G::SL)] = acc[k] * scale;
}

// The separable log-gain gradients' partial sums over one middle tile
// (f = hi * 2^A + run * 2^R + e), p = dG * G in layout R = 5 (register k holds
// hi bits 0-4, lane bits 0-4 hold e, the thread's higher bits hi bits 5 and
// up).  With R <= log2 C = cbits <= A, e is channel bits 0-4, the run's low
// qb = cbits - 5 bits are the channel group q, and a row hi of the tile is
// one token n = f >> cbits.  p goes through the tile's LDS in natural [hi][e]
// order (the exchanges are over), then
//   rows: thread tau adds row hi = tau's 32 elements, stored contiguously per
//         workgroup to rowpart[chunk][q][run >> qb][hi]
//         (sep_fused_final_kernel puts the rows in token order);
//   columns: thread tau adds column e = tau mod 32 over 32 rows, the groups
//         are added in `red`, to colpart[c][chunk][run >> qb].
// Fixed order throughout; registers stay as few as for storing dG.
template <int A, int HB, int R>
__device__ __forceinline__ void sep_tile_sums(const float (&p)[V], float *lds, float *red,
                                              uint32_t tau, uint32_t run, uint32_t chunk,
                                              uint32_t nchunks, uint32_t cbits,
                                              float *__restrict__ rowpart,
                                              float *__restrict__ colpart)
{
    constexpr uint32_t NG = 1u << (HB - 5);   // groups of 32 rows
    const uint32_t qb = cbits - R;
    const uint32_t q = run & ((1u << qb) - 1u);
    const uint32_t base = layout_base<R>(tau);
    __syncthreads();   // every thread's last reads of the tile exchanges are done
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pad(base + ((uint32_t)k << R))] = p[k];
    __syncthreads();
    float rs = 0.0f;
#pragma unroll
    for (uint32_t e = 0; e < 32u; ++e)
        rs += lds[pad((tau << R) + e)];
    const size_t rblock = ((size_t)((chunk << qb) | q) << (A - cbits)) | (run >> qb);
    rowpart[(rblock << HB) + tau] = rs;
    float cs = 0.0f;
    const uint32_t g = tau >> 5, e = tau & 31u;
#pragma unroll
    for (uint32_t i = 0; i < 32u; ++i)
        cs += lds[pad((((g << 5) + i) << R) + e)];
    red[g * 32u + e] = cs;
    __syncthreads();
    if (tau < 32u) {
        float t = 0.0f;
#pragma unroll
        for (uint32_t w = 0; w < NG; ++w)
            t += red[w * 32u + tau];
        const uint32_t c = (q << R) | tau;
        const uint32_t np = nchunks << (A - cbits);
        colpart[(size_t)c * np + ((chunk << (A - cbits)) | (run >> qb))] = t;
    }
}

// The same sums in the one-slice-per-chunk form (SINGLE, 2^15-element tiles),
// which does not hold the gain: d = dG in the tile's LDS, and since
// G[n][c] = exp(g_t[n]) exp(g_c[c]) the row sum is exp(g_t[n]) times the
// sum of d exp(g_c[c]) and the column sum exp(g_c[c]) times the sum of
// d exp(g_t[n]); both factors come from small LDS tables (the tile's 32
// channels, its 2^HB rows).  Products are stored to LDS as they are formed,
// so this needs no register array beyond the two tiles.
template <int A, int HB, int R>
__device__ __forceinline__ void sep_tile_sums_single(
    const float (&vx)[V], const float (&vd)[V], float scale, float *lds, float *red, float *egc,
    float *egt, const float *__restrict__ gt, const float *__restrict__ gc, uint32_t tau,
    uint32_t run, uint32_t chunk, uint32_t nchunks, uint32_t cbits, float *__restrict__ rowpart,
    float *__restrict__ colpart)
{
    constexpr uint32_t NG = 1u << (HB - 5);
    const uint32_t qb = cbits - R;
    const uint32_t q = run & ((1u << qb) - 1u);
    const uint32_t rl = run >> qb;
    const uint32_t base = layout_base<R>(tau);
    __syncthreads();   // every thread's last reads of the tile exchanges are done
#pragma unroll
    for (int k = 0; k < V; ++k)
        lds[pad(base + ((uint32_t)k << R))] = vx[k] * vd[k] * scale;
    if (tau < 32u)
        egc[tau] = __expf(gc[(q << R) | tau]);
    egt[tau] = __expf(gt[((size_t)tau << (A - cbits)) | rl]);   // row hi = tau: token n
    __syncthreads();
    float rs = 0.0f;
#pragma unroll
    for (uint32_t e = 0; e < 32u; ++e)
        rs += lds[pad((tau << R) + e)] * egc[e];
    const size_t rblock = ((size_t)((chunk << qb) | q) << (A - cbits)) | rl;
    rowpart[(rblock << HB) + tau] = rs * egt[tau];
    float cs = 0.0f;
    const uint32_t g = tau >> 5, e = tau & 31u;
#pragma unroll
    for (uint32_t i = 0; i < 32u; ++i)
        cs += lds[pad((((g << 5) + i) << R) + e)] * egt[(g << 5) + i];
    red[g * 32u + e] = cs;
    __syncthreads();
    if (tau < 32u) {
        float t = 0.0f;
#pragma unroll
        for (uint32_t w = 0; w < NG; ++w)
            t += red[w * 32u + tau];
        const uint32_t c = (q << R) | tau;
        const uint32_t np = nchunks << (A - cbits);
        colpart[(size_t)c * np + ((chunk << (A - cbits)) | rl)] = t * egc[tau];
    }
    __syncthreads();   // the tile's LDS is free again for the inverse exchanges
}

// Three-pass dG and dX together.  After OUTER_FWD of x and dy (one launch),
// one workgroup owns one workspace run for a chunk of slices.  For each slice
// it transforms both tiles over the HB high bits, so both are now transformed
// over every bit, and accumulates their product; it then finishes dY's mixer
// on the same tile (gain, inverse over the HB bits) and stores it back in
// place for OUTER_INV, which writes dX.  dY's transform is computed once for
// both gradients.
//
// With several slices per chunk the product sum keeps this kernel at one
// workgroup per CU (it holds the sum, the gain and both tiles: about 200
// registers), so the loads of the next slice are issued early instead of
// relying on other workgroups to cover their latency: x's as soon as x's tile
// has been used, dy's right after the store of the current one.  With one
// slice per chunk (SINGLE) the product is stored as soon as it is formed and
// the gain is read after it, when x's tile is dead; 2^15-element tiles (1024
// threads, at most 128 registers) always take this form.
//
// MIX_X: x's tile also goes through the gain and the inverse and is stored
// back to wsx (the forward mixer's middle pass on x, for the block's backward,
// which needs Z' as well), after the product and before the next slice's load.
//
// SEPSUM (separable gains, R = 5, HB >= 6, R <= log2 C <= A): instead of
// storing dG the workgroup forms the two log-gain gradients' partial sums of
// dG * G over its tile and writes them to rowpart / colpart (sep_tile_sums
// with several slices per chunk, sep_tile_sums_single with one).
template <int A, int HB, int R, class Gain, bool SINGLE, bool MIX_X = false, bool SEPSUM = false>
__global__ void __launch_bounds__(1 << (HB + R - VB))
grad_mix_middle_kernel(float *__restrict__ wsx, float *__restrict__ wsd, Gain gain,
                       float *__restrict__ out, uint32_t nslices, uint32_t per_chunk,
                       float *__restrict__ rowpart, float *__restrict__ colpart, uint32_t cbits)
{
    constexpr int M = HB + R;
    using G = Groups<M, R>;
    using GM = GainMap<A, R>;
    constexpr float scale = 1.0f / (float)(1u << (A + HB));
    __shared__ float lds[pad(1u << M)];
    const uint32_t tau = threadIdx.x;
    const uint32_t run = blockIdx.x & ((1u << (A - R)) - 1u);
    const uint32_t chunk = blockIdx.x >> (A - R);
    const uint32_t b0 = chunk * per_chunk;
    const uint32_t b1 = min(b0 + per_chunk, nslices);
    const auto tile = [&](const float *ws, uint32_t b) {
        return buffer(ws + ((size_t)b << (A + HB)) + ((size_t)run << M), (1u << M) * 4u);
    };
    static_assert(!SEPSUM || (R == VB && G::SL == R && HB >= 6),
                  "the fused separable sums take the product in layout R = 5");
    float *o = SEPSUM ? out
                      : out + ((size_t)chunk << (A + HB)) + ((size_t)run << R) +
                            GM::at(layout_base<G::SL>(tau));
    float vx[V], vd[V];
    load_layout<G::TOP, ContigMap, float>(vx, tile(wsx, b0), tau);
    load_layout<G::TOP, ContigMap, float>(vd, tile(wsd, b0), tau);
    if constexpr (SINGLE) {
        butterflies<G::JT, VB>(vx);
        butterflies<G::JT, VB>(vd);
        forward_groups<M, R, 0, G::TOP, true>(lds, vx, tau);
        forward_groups<M, R, 0, G::TOP, true>(lds, vd, tau);
        if constexpr (SEPSUM && std::is_same_v<Gain, LogSeparableGain>) {
            __shared__ float red[32u << (HB - 5)], egt[1u << HB], egc[32];
            sep_tile_sums_single<A, HB, R>(vx, vd, scale, lds, red, egc, egt, gain.gt, gain.gc,
                                           tau, run, chunk, gridDim.x >> (A - R), cbits,
                                           rowpart, colpart);
        } else {
#pragma unroll
            for (int k = 0; k < V; ++k)
                o[GM::at((uint32_t)k << G::SL)] = vx[k] * vd[k] * scale;
        }
        __builtin_amdgcn_sched_barrier(0);   // keep the gain loads after the product
        float gv[V];
        gain.template load<G::SL, GM, true>(gv, run << R, tau);
        if constexpr (MIX_X) {
            apply_gain<A + HB>(vx, gv);
            if constexpr (G::NBOT > 0)
                inverse_groups<M, R, G::NBOT - 1>(lds, vx, tau);
            butterflies<G::JT, VB>(vx);
            store_layout<G::TOP, ContigMap, float>(vx, tile(wsx, b0), tau);
        }
        apply_gain<A + HB>(vd, gv);
        if constexpr (G::NBOT > 0)
            inverse_groups<M, R, G::NBOT - 1>(lds, vd, tau);
        butterflies<G::JT, VB>(vd);
        store_layout<G::TOP, ContigMap, float>(vd, tile(wsd, b0), tau);
    } else {
        float acc[V], gv[V];
#pragma unroll
        for (int k = 0; k < V; ++k)
            acc[k] = 0.0f;
        gain.template load<G::SL, GM, true>(gv, run << R, tau);   // the same for every slice
        for (uint32_t b = b0; b < b1; ++b) {   // uniform over the workgroup
            const bool more = b + 1 < b1;
            butterflies<G::JT, VB>(vx);
            butterflies<G::JT, VB>(vd);
            forward_groups<M, R, 0, G::TOP, true>(lds, vx, tau);
            forward_groups<M, R, 0, G::TOP, true>(lds, vd, tau);
#pragma unroll
            for (int k = 0; k < V; ++k)
                acc[k] = fmaf(vx[k], vd[k], acc[k]);
            if constexpr (MIX_X) {
                apply_gain<A + HB>(vx, gv);
                if constexpr (G::NBOT > 0)
                    inverse_groups<M, R, G::NBOT - 1>(lds, vx, tau);
                butterflies<G::JT, VB>(vx);
                store_layout<G::TOP, ContigMap, float>(vx, tile(wsx, b), tau);
            }
            if (more)
                load_layout<G::TOP, ContigMap, float>(vx, tile(wsx, b + 1), tau);
            apply_gain<A + HB>(vd, gv);
            if constexpr (G::NBOT > 0)
                inverse_groups<M, R, G::NBOT - 1>(lds, vd, tau);
            butterflies<G::JT, VB>(vd);
            store_layout<G::TOP, ContigMap, float>(vd, tile(wsd, b), tau);
            if (more)
                load_layout<G::TOP, ContigMap, float>(vd, tile(wsd, b + 1), tau);
        }
        if constexpr (SEPSUM) {
            float p[V];
#pragma unroll
            for (int k = 0; k < V; ++k)
                p[k] = acc[k] * scale * gv[k];
            __shared__ float red[32u << (HB > 5 ? HB - 5 : 0)];
            sep_tile_sums<A, HB, R>(p, lds, red, tau, run, chunk, gridDim.x >> (A - R), cbits,
                                    rowpart, colpart);
        } else {
#pragma unroll
            for (int k = 0; k < V; ++k)
                o[GM::at((uint32_t)k << G::SL)] = acc[k] * scale;
        }
    }
}

// Fused dG (2^11 <= L <= 2^15): one workgroup per chunk of slices, each
// slice transformed whole.
template <int K, typename T>
__global__ void __launch_bounds__(1 << (K - VB))
grad_fused_kernel(const T *__restrict__ x, const T *__restrict__ dy, float *__restrict__ out,
                  uint32_t nslices, uint32_t per_chunk, uint32_t nvalid)
{
    using G = Groups<K, 0>;
    __shared__ float lds[pad(1u << K)];
    const uint32_t tau = threadIdx.x;
    const uint32_t chunk = blockIdx.x;
    const uint32_t b0 = chunk * per_chunk;
    const uint32_t b1 = min(b0 + per_chunk, nslices);
    float acc[V];
#pragma unroll
    for (int k = 0; k < V; ++k)
        acc[k] = 0.0f;
    for (uint32_t b = b0; b < b1; ++b) {
        float vx[V], vd[V];
        load_tile<G::TOP, K, T>(vx, x + (size_t)b * nvalid, nvalid, tau);
        load_tile<G::TOP, K, T>(vd, dy + (size_t)b * nvalid, nvalid, tau);
        butterflies<G::JT, VB>(vx);
        butterflies<G::JT, VB>(vd);
        forward_groups<K, 0, 0, G::TOP, true>(lds, vx, tau);
        forward_groups<K, 0, 0, G::TOP, true>(lds, vd, tau);
#pragma unroll
        for (int k = 0; k < V; ++k)
            acc[k] = fmaf(vx[k], vd[k], acc[k]);
    }
    constexpr float scale = 1.0f / (float)(1u << K);
    float *o = out + ((size_t)chunk << K) + layout_base<G::SL>(tau);
#pragma unroll
    for (int k = 0; k < V; ++k)
        o[(uint32_t)k << G::SL] = acc[k] * scale;
}

// In-place unnormalised butterfly of the L values in LDS (all threads).
__device__ void lds_fwht(float *s, int L)
{
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
}

__device__ __forceinline__ float widen(float v) { return v; }
__device__ __forceinline__ float widen(__bf16 v) { return (float)v; }

// Small dG (L <= 2^10): one 256-thread workgroup per chunk, stages in LDS.
template <typename T>
__global__ void __launch_bounds__(256)
grad_small_kernel(const T *__restrict__ x, const T *__restrict__ dy, float *__restrict__ out,
                  int K, uint32_t nslices, uint32_t per_chunk, uint32_t nvalid)
{
    __shared__ float sx[1 << kMaxSmall], sd[1 << kMaxSmall], acc[1 << kMaxSmall];
    const int L = 1 << K;
    const uint32_t chunk = blockIdx.x;
    const uint32_t b0 = chunk * per_chunk;
    const uint32_t b1 = min(b0 + per_chunk, nslices);
    for (int i = threadIdx.x; i < L; i += blockDim.x)
        acc[i] = 0.0f;
    for (uint32_t b = b0; b < b1; ++b) {
        __syncthreads();
        const size_t base = (size_t)b * nvalid;
        for (int i = threadIdx.x; i < L; i += blockDim.x) {
            sx[i] = (uint32_t)i < nvalid ? widen(x[base + i]) : 0.0f;
            sd[i] = (uint32_t)i < nvalid ? widen(dy[base + i]) : 0.0f;
        }
        lds_fwht(sx, L);
        lds_fwht(sd, L);
        for (int i = threadIdx.x; i < L; i += blockDim.x)
            acc[i] = fmaf(sx[i], sd[i], acc[i]);
    }
    __syncthreads();
    const float scale = 1.0f / (float)L;
    for (int i = threadIdx.x; i < L; i += blockDim.x)
        out[((size_t)chunk << K) + i] = acc[i] * scale;
}

// out[f] = sum over chunks of part[chunk][f], in chunk order.  Four floats
// per thread when L is a multiple of 4 (both buffers are 16-byte aligned),
// else (L = 1 or 2) one.
__global__ void __launch_bounds__(256)
sum_chunks_kernel(const float *__restrict__ part, float *__restrict__ out, uint64_t L,
                  uint32_t nchunks)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    const uint64_t i0 = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x;
    if (L % 4 != 0) {
        for (uint64_t f = i0; f < L; f += stride) {
            float s = part[f];
            for (uint32_t c = 1; c < nchunks; ++c)
                s += part[c * L + f];
            out[f] = s;
        }
        return;
    }
    const uint64_t n4 = L / 4;
    const float4 *p4 = reinterpret_cast<const float4 *>(part);
    float4 *o4 = reinterpret_cast<float4 *>(out);
    for (uint64_t i = i0; i < n4; i += stride) {
        float4 s = p4[i];
        for (uint32_t c = 1; c < nchunks; ++c) {
            const float4 v = p4[c * n4 + i];
            s.x += v.x;
            s.y += v.y;
            s.z += v.z;
            s.w += v.w;
        }
        o4[i] = s;
    }
}

__global__ void __launch_bounds__(256)
fill_zero_kernel(float *__restrict__ out, uint64_t n)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; i < n; i += stride)
        out[i] = 0.0f;
}

// dg_t[n] = sum_c dG[n][c] exp(g_t[n] + g_c[c]); one wavefront per row n.
__global__ void __launch_bounds__(256)
sep_rows_kernel(const float *__restrict__ dG, const float *__restrict__ gt,
                const float *__restrict__ gc, float *__restrict__ dgt, uint32_t P, uint32_t cbits)
{
    const uint32_t C = 1u << cbits;
    const uint32_t row = blockIdx.x * 4u + (threadIdx.x >> 6);
    const uint32_t lane = threadIdx.x & 63u;
    if (row >= P)
        return;   // whole wavefront (no barriers in this kernel)
    const float g = gt[row];
    const float *d = dG + (size_t)row * C;
    float s = 0.0f;
    for (uint32_t c = lane; c < C; c += 64)
        s = fmaf(d[c], __expf(g + gc[c]), s);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        s += __shfl_down(s, off, 64);
    if (lane == 0)
        dgt[row] = s;
}

// Sum of the 256 values in red[] (fixed tree order); result in red[0].
__device__ __forceinline__ void block_sum_256(float *red)
{
    for (int w = 128; w > 0; w >>= 1) {
        __syncthreads();
        if ((int)threadIdx.x < w)
            red[threadIdx.x] += red[threadIdx.x + w];
    }
    __syncthreads();
}

// Column partial sums of dG*G over a block of rows.  Block (strip, rblk)
// covers rows [rblk*RB, ...) and columns [strip*256, ...).  With C <= 256 the
// 256 threads hold 256/C rows of the C columns per step and their sums per
// column are added in LDS; with C > 256 each thread owns one column of the
// strip.  part[c][rblk] receives the block's sums (column-major, so that
// the final sum over row blocks reads each column contiguously).
__global__ void __launch_bounds__(256)
sep_cols_partial_kernel(const float *__restrict__ dG, const float *__restrict__ gt,
                        const float *__restrict__ gc, float *__restrict__ part, uint32_t P,
                        uint32_t cbits, uint32_t rows_per_block)
{
    __shared__ float red[256];
    const uint32_t C = 1u << cbits;
    const uint32_t tid = threadIdx.x;
    const uint32_t r0 = blockIdx.x * rows_per_block;
    const uint32_t r1 = min(r0 + rows_per_block, P);
    const uint32_t cw = C < 256u ? C : 256u;              // columns per step
    const uint32_t c = blockIdx.y * 256u + (tid & (cw - 1u));
    const uint32_t rstep = 256u / cw;
    float s = 0.0f;
    if (tid < rstep * cw) {
        const float gcc = gc[c];
#pragma unroll 8
        for (uint32_t r = r0 + tid / cw; r < r1; r += rstep)
            s = fmaf(dG[(size_t)r * C + c], __expf(gt[r] + gcc), s);
    }
    red[tid] = s;
    __syncthreads();
    if (cw < 256u) {
        // add the rstep partial sums of each column: threads tid and tid + k*cw
        for (uint32_t w = 128u; w >= cw; w >>= 1) {
            if (tid < w)
                red[tid] += red[tid + w];
            __syncthreads();
        }
    }
    if (tid < cw)
        part[(size_t)c * gridDim.x + blockIdx.x] = red[tid];
}

// Row sums (dg_t) and column partial sums of dG*G in one pass over dG, for
// C = 2^CB <= 256.  Block blockIdx.x covers rows [r0, r0 + rows_per_block);
// a row's C columns spread over SEG = min(C, 64) lanes, KPL = C / SEG
// consecutive columns each (one 4-, 8- or 16-byte load), so a wave takes
// RPW = 64 / SEG rows at a time and a row sum is a segmented wave reduction
// with no LDS.  Each iteration issues the loads of U such row steps (the
// block's four waves interleaved) before using any: rows past the block
// load its last row again and add nothing, so no load sits in a branch that
// would make the wave wait for it.  Each exp is taken once.  The column sums
// of a wave's rows are added across the wave, then over the four waves in
// LDS: part[c][blockIdx.x] (column-major), fixed order throughout.
template <int CB>
__global__ void __launch_bounds__(256)
sep_rows_cols_kernel(const float *__restrict__ dG, const float *__restrict__ gt,
                     const float *__restrict__ gc, float *__restrict__ dgt,
                     float *__restrict__ part, uint32_t P, uint32_t rows_per_block)
{
    constexpr uint32_t C = 1u << CB;
    constexpr uint32_t SEG = C < 64u ? C : 64u;
    constexpr uint32_t RPW = 64u / SEG;
    constexpr uint32_t KPL = C / SEG;
    constexpr uint32_t U = 4;
    typedef float fvec __attribute__((ext_vector_type(KPL)));
    __shared__ float red[4][C];
    const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
    const uint32_t c0 = (lane & (SEG - 1u)) * KPL;   // first of the lane's KPL columns
    const uint32_t rw = lane / SEG;
    const uint32_t r0 = blockIdx.x * rows_per_block;
    const uint32_t r1 = min(r0 + rows_per_block, P);   // > r0: the grid covers P rows
    float gcv[KPL], cs[KPL];
#pragma unroll
    for (uint32_t k = 0; k < KPL; ++k) {
        gcv[k] = gc[c0 + k];
        cs[k] = 0.0f;
    }
    for (uint32_t rb = r0; rb < r1; rb += U * 4u * RPW) {   // uniform over the block
        float v[U][KPL], g[U];
#pragma unroll
        for (uint32_t u = 0; u < U; ++u) {
            const uint32_t r = min(rb + (u * 4u + wave) * RPW + rw, r1 - 1u);
            g[u] = gt[r];
            if constexpr (KPL == 1) {
                v[u][0] = dG[(size_t)r * C + c0];
            } else {
                const fvec q = *reinterpret_cast<const fvec *>(dG + (size_t)r * C + c0);
#pragma unroll
                for (uint32_t k = 0; k < KPL; ++k)
                    v[u][k] = q[k];
            }
        }
#pragma unroll
        for (uint32_t u = 0; u < U; ++u) {
            const uint32_t r = rb + (u * 4u + wave) * RPW + rw;
            const bool live = r < r1;
            float rs = 0.0f;
#pragma unroll
            for (uint32_t k = 0; k < KPL; ++k) {
                const float p = live ? v[u][k] * __expf(g[u] + gcv[k]) : 0.0f;
                cs[k] += p;
                rs += p;
            }
#pragma unroll
            for (uint32_t off = SEG >> 1; off > 0; off >>= 1)
                rs += __shfl_xor(rs, off, 64);
            if ((lane & (SEG - 1u)) == 0 && live)
                dgt[r] = rs;
        }
    }
#pragma unroll
    for (uint32_t k = 0; k < KPL; ++k) {
        float t = cs[k];
#pragma unroll
        for (uint32_t off = SEG; off < 64u; off <<= 1)
            t += __shfl_xor(t, off, 64);
        if (rw == 0)
            red[wave][c0 + k] = t;
    }
    __syncthreads();
    for (uint32_t c = threadIdx.x; c < C; c += 256u)
        part[(size_t)c * gridDim.x + blockIdx.x] =
            ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
}

// dgc[c] = sum over row blocks of part[c][b] (column-major: each block
// reads its column contiguously): one block per column, 256-way strided sums
// then a fixed-order tree.
__global__ void __launch_bounds__(256)
sep_cols_final_kernel(const float *__restrict__ part, float *__restrict__ dgc, uint32_t nblk)
{
    __shared__ float red[256];
    const uint32_t c = blockIdx.x;
    float s = 0.0f;
    for (uint32_t b = threadIdx.x; b < nblk; b += 256)
        s += part[(size_t)c * nblk + b];
    red[threadIdx.x] = s;
    block_sum_256(red);
    if (threadIdx.x == 0)
        dgc[c] = red[0];
}

// The fused separable sums' last step: blocks [0, nrowblk) give the row
// sums, i = rl * 2^HB + hi of rowpart[j][rl][hi] (j = chunk * Q + q, nq of
// them) going to token n = hi * 2^(A - cbits) + rl; the next C blocks
// dgc[c] = sum over colpart[c][0 .. np).  Fixed order.
__global__ void __launch_bounds__(256)
sep_fused_final_kernel(const float *__restrict__ rowpart, const float *__restrict__ colpart,
                       float *__restrict__ dgt, float *__restrict__ dgc, uint32_t P, uint32_t nq,
                       uint32_t np, uint32_t nrowblk, uint32_t hb, uint32_t rlbits)
{
    __shared__ float red[256];
    if (blockIdx.x < nrowblk) {   // uniform per block
        const uint32_t i = blockIdx.x * 256u + threadIdx.x;
        if (i < P) {
            float s = 0.0f;
            for (uint32_t j = 0; j < nq; ++j)
                s += rowpart[(size_t)j * P + i];
            dgt[((i & ((1u << hb) - 1u)) << rlbits) | (i >> hb)] = s;
        }
        return;
    }
    const uint32_t c = blockIdx.x - nrowblk;
    float s = 0.0f;
    for (uint32_t b = threadIdx.x; b < np; b += 256u)
        s += colpart[(size_t)c * np + b];
    red[threadIdx.x] = s;
    block_sum_256(red);
    if (threadIdx.x == 0)
        dgc[c] = red[0];
}

inline hipError_t record(hipEvent_t ev, hipStream_t st)
{
    return ev ? hipEventRecord(ev, st) : hipSuccess;
}

inline uint32_t grid_for(uint64_t n)
{
    const uint64_t g = (n + 255) / 256;
    return (uint32_t)(g < 4096 ? (g ? g : 1) : 4096);
}

// dG (2^-K-scaled sum over the batch) into `dst` ([2^K] floats).
template <int K, typename T>
hipError_t grad_three_pass(const T *x, const T *dy, float *dst, const BackwardArgs &a,
                           const BackwardLayout &lay)
{
    constexpr Split sp = three_pass_split(K);
    constexpr int A = sp.A, HB = sp.HB, R = sp.R;
    const hipStream_t st = a.stream;
    float *wsx = a.ws + lay.wsx;
    float *wsd = a.ws + lay.wsd;
    hipError_t e;
    if ((e = launch_outer_fwd<K, T>(x, wsx, a.B, a.nvalid, st)) != hipSuccess) return e;
    if ((e = launch_outer_fwd<K, T>(dy, wsd, a.B, a.nvalid, st)) != hipSuccess) return e;
    float *o = lay.nchunks > 1 ? a.ws + lay.part : dst;
    hipLaunchKernelGGL((grad_middle_kernel<A, HB, R>), dim3(lay.nchunks << (A - R)),
                       dim3(1u << (HB + R - VB)), 0, st, wsx, wsd, o, (uint32_t)a.B,
                       lay.per_chunk);
    return hipGetLastError();
}

template <int K, typename T>
hipError_t grad_fused(const T *x, const T *dy, float *dst, const BackwardArgs &a,
                      const BackwardLayout &lay)
{
    float *o = lay.nchunks > 1 ? a.ws + lay.part : dst;
    hipLaunchKernelGGL((grad_fused_kernel<K, T>), dim3(lay.nchunks), dim3(1u << (K - VB)), 0,
                       a.stream, x, dy, o, (uint32_t)a.B, lay.per_chunk, a.nvalid);
    return hipGetLastError();
}

template <typename T>
hipError_t grad_dispatch(const BackwardArgs &a, const BackwardLayout &lay, float *dst)
{
    const T *x = static_cast<const T *>(a.x);
    const T *dy = static_cast<const T *>(a.dy);
    hipError_t e = hipSuccess;
    if (a.plan == PLAN_SMALL) {
        float *o = lay.nchunks > 1 ? a.ws + lay.part : dst;
        hipLaunchKernelGGL((grad_small_kernel<T>), dim3(lay.nchunks), dim3(256), 0, a.stream, x,
                           dy, o, a.K, (uint32_t)a.B, lay.per_chunk, a.nvalid);
        e = hipGetLastError();
    } else if (a.plan == PLAN_FUSED) {
        switch (a.K) {
#define WHTMIX_GF_CASE(k) \
    case k: e = grad_fused<k, T>(x, dy, dst, a, lay); break;
            WHTMIX_GF_CASE(11) WHTMIX_GF_CASE(12) WHTMIX_GF_CASE(13) WHTMIX_GF_CASE(14)
            WHTMIX_GF_CASE(15)
#undef WHTMIX_GF_CASE
        default: return hipErrorInvalidValue;
        }
    } else {
        switch (a.K) {
#define WHTMIX_G3_CASE(k) \
    case k: e = grad_three_pass<k, T>(x, dy, dst, a, lay); break;
            WHTMIX_G3_CASE(12) WHTMIX_G3_CASE(13) WHTMIX_G3_CASE(14) WHTMIX_G3_CASE(15)
            WHTMIX_G3_CASE(16) WHTMIX_G3_CASE(17) WHTMIX_G3_CASE(18) WHTMIX_G3_CASE(19)
            WHTMIX_G3_CASE(20) WHTMIX_G3_CASE(21) WHTMIX_G3_CASE(22) WHTMIX_G3_CASE(23)
            WHTMIX_G3_CASE(24) WHTMIX_G3_CASE(25) WHTMIX_G3_CASE(26) WHTMIX_G3_CASE(27)
            WHTMIX_G3_CASE(28) WHTMIX_G3_CASE(29) WHTMIX_G3_CASE(30)
#undef WHTMIX_G3_CASE
        default: return hipErrorInvalidValue;
        }
    }
    if (e != hipSuccess || lay.nchunks <= 1) return e;
    const uint64_t L = uint64_t(1) << a.K;
    hipLaunchKernelGGL(sum_chunks_kernel, dim3(grid_for(L)), dim3(256), 0, a.stream,
                       a.ws + lay.part, dst, L, lay.nchunks);
    return hipGetLastError();
}

}  // namespace

BackwardLayout backward_layout(int plan, int K, int64_t B, int64_t C, bool separable)
{
    BackwardLayout lay{};
    const uint64_t L = uint64_t(1) << K;
    uint64_t cursor = 0;
    if (plan == PLAN_THREE_PASS) {
        lay.wsx = cursor;
        cursor += (uint64_t)B * L;
        lay.wsd = cursor;
        cursor += (uint64_t)B * L;
    }
    uint64_t want;
    if (plan == PLAN_THREE_PASS) {
        const Split sp = three_pass_split(K);
        // about two workgroups per CU over the chunks and runs (the fused
        // kernel holds one CU each); one slice per chunk for 2^15 tiles
        const uint64_t runs = uint64_t(1) << (sp.A - sp.R);
        want = sp.HB + sp.R == kMaxTile ? (uint64_t)B : (512 + runs - 1) / runs;
    } else {
        want = plan == PLAN_FUSED ? 1024 : 2048;
    }
    uint64_t nch = B < 1 ? 1 : ((uint64_t)B < want ? (uint64_t)B : want);
    const uint64_t per = ((uint64_t)B + nch - 1) / nch;
    nch = B < 1 ? 1 : ((uint64_t)B + per - 1) / per;
    lay.per_chunk = (uint32_t)(per ? per : 1);
    lay.nchunks = (uint32_t)nch;
    if (lay.nchunks > 1) {
        lay.part = cursor;
        cursor += (uint64_t)lay.nchunks * L;
    }
    if (separable) {
        const uint64_t P = L / (uint64_t)C;
        lay.dg = cursor;
        cursor += L;
        // about 2048 row blocks (the single-pass kernel's workgroups), at least
        // one step of its rows: 256 / min(C, 64)
        uint64_t rpb = (P + 2047) / 2048;
        const uint64_t step = 256 / (C < 64 ? (uint64_t)C : 64);
        if (rpb < step) rpb = step;
        lay.rows_per_block = (uint32_t)rpb;
        lay.col_blocks = (uint32_t)((P + rpb - 1) / rpb);
        lay.colpart = cursor;
        cursor += (uint64_t)lay.col_blocks * (uint64_t)C;
    }
    int cbits = 0;
    while ((int64_t(1) << cbits) < C) ++cbits;
    if (separable && plan == PLAN_THREE_PASS) {
        // where the middle pass can, it forms the partial sums itself
        // (grad_mix_middle_kernel SEPSUM; the paths that store dG use the
        // regions above): rows [chunk][C / 2^R][P], columns
        // [C][chunk][2^(A - cbits)]
        const Split sp = three_pass_split(K);
        if (sp.R == VB && sp.HB >= 6 && sp.HB + sp.R <= kMaxTile && cbits >= sp.R &&
            cbits <= sp.A) {
            lay.sep_fused = 1;
            lay.rowpart = cursor;
            cursor += (uint64_t)lay.nchunks * (L >> sp.R);
            lay.fcolpart = cursor;
            cursor += (uint64_t)C * ((uint64_t)lay.nchunks << (sp.A - cbits));
        }
    }
    // The dX pass runs after dG and reuses the start of the workspace.
    const uint64_t fwd = plan == PLAN_THREE_PASS ? (uint64_t)B * L : 0;
    lay.floats = cursor > fwd ? cursor : fwd;
    return lay;
}

namespace {

// The single-pass row / column reduction covers C <= 2^8; wider C keeps the
// separate row and column kernels.
constexpr int kSepFusedMaxCbits = 8;

// Separable log-gain gradients from the joint dG in dst:
// dg_t = row sums and dg_c = column sums of dG o G.
hipError_t separable_reductions(const BackwardArgs &a, const BackwardLayout &lay, const float *dst)
{
    const hipStream_t st = a.stream;
    const uint64_t L = uint64_t(1) << a.K;
    const uint32_t P = (uint32_t)(L >> a.cbits);
    const uint32_t C = 1u << a.cbits;
    hipError_t e;
    if (a.cbits <= kSepFusedMaxCbits) {
        // one pass: row sums and column partials together
        const dim3 grid(lay.col_blocks), block(256);
        float *colpart = a.ws + lay.colpart;
        switch (a.cbits) {
#define WHTMIX_SEP_CASE(cb)                                                                    \
    case cb:                                                                                  \
        hipLaunchKernelGGL(sep_rows_cols_kernel<cb>, grid, block, 0, st, dst, a.gain_t,       \
                           a.gain_c, a.dgt, colpart, P, lay.rows_per_block);                  \
        break;
            WHTMIX_SEP_CASE(0) WHTMIX_SEP_CASE(1) WHTMIX_SEP_CASE(2) WHTMIX_SEP_CASE(3)
            WHTMIX_SEP_CASE(4) WHTMIX_SEP_CASE(5) WHTMIX_SEP_CASE(6) WHTMIX_SEP_CASE(7)
            WHTMIX_SEP_CASE(8)
#undef WHTMIX_SEP_CASE
        default: return hipErrorInvalidValue;
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
        hipLaunchKernelGGL(sep_rows_kernel, dim3((P + 3) / 4), dim3(256), 0, st, dst, a.gain_t,
                           a.gain_c, a.dgt, P, (uint32_t)a.cbits);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(sep_cols_partial_kernel, dim3(lay.col_blocks, C / 256u), dim3(256), 0,
                           st, dst, a.gain_t, a.gain_c, a.ws + lay.colpart, P, (uint32_t)a.cbits,
                           lay.rows_per_block);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(sep_cols_final_kernel, dim3(C), dim3(256), 0, st, a.ws + lay.colpart,
                       a.dgc, lay.col_blocks);
    return hipGetLastError();
}

// Calls f with the streamed form of a joint gain (other gains unchanged).
template <class Gain, class F>
inline hipError_t with_streamed_gain(Gain gain, F &&f)
{
    return f(gain);
}
template <class F>
inline hipError_t with_streamed_gain(FullGain gain, F &&f)
{
    return f(StreamedGain{gain.g});
}

// The fused middle on the outer transforms in wsx and wsd (dG, and dY's mixer
// up to its last pass, in place in wsd) -> [chunk sums] -> [separable sums].
template <int K, class Gain, bool MIX_X = false>
hipError_t grad_middle_phase(const BackwardArgs &a, const BackwardLayout &lay, float *dst,
                             Gain gain)
{
    constexpr Split sp = three_pass_split(K);
    constexpr int A = sp.A, HB = sp.HB, R = sp.R;
    const hipStream_t st = a.stream;
    float *wsx = a.ws + lay.wsx;
    float *wsd = a.ws + lay.wsd;
    hipError_t e;
    if constexpr (std::is_same_v<Gain, LogSeparableGain> && R == VB && HB >= 6 &&
                  HB + R <= kMaxTile) {
        if (lay.sep_fused) {
            // the middle pass forms the row and column partial sums of dG * G
            // (the several-slices form up to 2^14-element tiles, any slices
            // per chunk; the one-slice form for 2^15), then one small kernel
            // adds them up
            constexpr bool single = HB + R == kMaxTile;
            hipLaunchKernelGGL((grad_mix_middle_kernel<A, HB, R, Gain, single, MIX_X, true>),
                               dim3(lay.nchunks << (A - R)), dim3(1u << (HB + R - VB)), 0, st,
                               wsx, wsd, gain, nullptr, (uint32_t)a.B, lay.per_chunk,
                               a.ws + lay.rowpart, a.ws + lay.fcolpart, (uint32_t)a.cbits);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            const uint32_t P = (uint32_t)((uint64_t(1) << K) >> a.cbits);
            const uint32_t nrowblk = (P + 255u) / 256u;
            hipLaunchKernelGGL(sep_fused_final_kernel, dim3(nrowblk + (1u << a.cbits)),
                               dim3(256), 0, st, a.ws + lay.rowpart, a.ws + lay.fcolpart, a.dgt,
                               a.dgc, P, lay.nchunks << (a.cbits - R),
                               lay.nchunks << (A - a.cbits), nrowblk, (uint32_t)HB,
                               (uint32_t)(A - a.cbits));
            return hipGetLastError();
        }
    }
    float *o = lay.nchunks > 1 ? a.ws + lay.part : dst;
    if (lay.per_chunk == 1) {
        e = with_middle_gain(gain, a.B, [&](auto g) {
            hipLaunchKernelGGL((grad_mix_middle_kernel<A, HB, R, decltype(g), true, MIX_X>),
                               dim3(lay.nchunks << (A - R)), dim3(1u << (HB + R - VB)), 0, st,
                               wsx, wsd, g, o, (uint32_t)a.B, 1u, nullptr, nullptr, 0u);
            return hipGetLastError();
        });
        if (e != hipSuccess) return e;
    } else if constexpr (HB + R < kMaxTile) {
        // each workgroup reads its run's gain once and holds it for the chunk's
        // slices: a joint gain streams (non-temporal), so it does not displace
        // the two workspaces
        e = with_streamed_gain(gain, [&](auto g) {
            hipLaunchKernelGGL((grad_mix_middle_kernel<A, HB, R, decltype(g), false, MIX_X>),
                               dim3(lay.nchunks << (A - R)), dim3(1u << (HB + R - VB)), 0, st,
                               wsx, wsd, g, o, (uint32_t)a.B, lay.per_chunk, nullptr, nullptr,
                               0u);
            return hipGetLastError();
        });
        if (e != hipSuccess) return e;
    } else {
        return hipErrorInvalidValue;   // backward_layout gives 2^15 tiles one slice per chunk
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (lay.nchunks > 1) {
        const uint64_t L = uint64_t(1) << K;
        hipLaunchKernelGGL(sum_chunks_kernel, dim3(grid_for(L)), dim3(256), 0, st,
                           a.ws + lay.part, dst, L, lay.nchunks);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (a.gain_kind == GAIN_LOG_SEPARABLE &&
        (e = separable_reductions(a, lay, dst)) != hipSuccess)
        return e;
    return hipSuccess;
}

// Both gradients with the three-pass plan, sharing dY's transform:
//   OUTER_FWD of x and dy (one launch) -> the fused middle phase -> OUTER_INV (dX).
template <int K, typename T, class Gain>
hipError_t fused_three_pass(const BackwardArgs &a, const BackwardLayout &lay, float *dst,
                            Gain gain)
{
    const hipStream_t st = a.stream;
    float *wsx = a.ws + lay.wsx;
    float *wsd = a.ws + lay.wsd;
    hipError_t e = launch_outer_fwd2<K, T>(static_cast<const T *>(a.x),
                                           static_cast<const T *>(a.dy), wsx, wsd, a.B,
                                           a.nvalid, st);
    if (e != hipSuccess) return e;
    if ((e = grad_middle_phase<K, Gain>(a, lay, dst, gain)) != hipSuccess) return e;
    if ((e = record(a.events[1], st)) != hipSuccess) return e;
    return launch_outer_inv<K, T>(wsd, static_cast<T *>(a.dx), a.B, a.nvalid, st);
}

template <class Gain>
hipError_t middle_phase_dispatch(const BackwardArgs &a, const BackwardLayout &lay, float *dst,
                                 Gain gain)
{
    switch (a.K) {
#define WHTMIX_GM_CASE(k) \
    case k: return grad_middle_phase<k, Gain, true>(a, lay, dst, gain);
        WHTMIX_GM_CASE(12) WHTMIX_GM_CASE(13) WHTMIX_GM_CASE(14) WHTMIX_GM_CASE(15)
        WHTMIX_GM_CASE(16) WHTMIX_GM_CASE(17) WHTMIX_GM_CASE(18) WHTMIX_GM_CASE(19)
        WHTMIX_GM_CASE(20) WHTMIX_GM_CASE(21) WHTMIX_GM_CASE(22) WHTMIX_GM_CASE(23)
        WHTMIX_GM_CASE(24) WHTMIX_GM_CASE(25) WHTMIX_GM_CASE(26) WHTMIX_GM_CASE(27)
        WHTMIX_GM_CASE(28)
#undef WHTMIX_GM_CASE
    default: return hipErrorInvalidValue;
    }
}

template <typename T, class Gain>
hipError_t fused_dispatch(const BackwardArgs &a, const BackwardLayout &lay, float *dst, Gain gain)
{
    switch (a.K) {
#define WHTMIX_FB_CASE(k) \
    case k: return fused_three_pass<k, T, Gain>(a, lay, dst, gain);
        WHTMIX_FB_CASE(12) WHTMIX_FB_CASE(13) WHTMIX_FB_CASE(14) WHTMIX_FB_CASE(15)
        WHTMIX_FB_CASE(16) WHTMIX_FB_CASE(17) WHTMIX_FB_CASE(18) WHTMIX_FB_CASE(19)
        WHTMIX_FB_CASE(20) WHTMIX_FB_CASE(21) WHTMIX_FB_CASE(22) WHTMIX_FB_CASE(23)
        WHTMIX_FB_CASE(24) WHTMIX_FB_CASE(25) WHTMIX_FB_CASE(26) WHTMIX_FB_CASE(27)
        WHTMIX_FB_CASE(28) WHTMIX_FB_CASE(29) WHTMIX_FB_CASE(30)
#undef WHTMIX_FB_CASE
    default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t fused_gain(const BackwardArgs &a, const BackwardLayout &lay, float *dst)
{
    if (a.gain_kind == GAIN_LOG_SEPARABLE)
        return fused_dispatch<T>(a, lay, dst,
                                 LogSeparableGain{a.gain_t, a.gain_c, (uint32_t)a.cbits});
    return fused_dispatch<T>(a, lay, dst, FullGain{a.gain});
}

}  // namespace

hipError_t launch_backward_middle(const BackwardArgs &a)
{
    const bool separable = a.gain_kind == GAIN_LOG_SEPARABLE;
    const bool want_dg = separable ? (a.dgt != nullptr && a.dgc != nullptr) : (a.dgain != nullptr);
    if (!want_dg || a.B < 1 || a.plan != PLAN_THREE_PASS)
        return hipErrorInvalidValue;
    const BackwardLayout lay = backward_layout(a.plan, a.K, a.B, int64_t(1) << a.cbits, separable);
    float *dst = separable ? a.ws + lay.dg : a.dgain;
    if (separable)
        return middle_phase_dispatch(a, lay, dst,
                                     LogSeparableGain{a.gain_t, a.gain_c, (uint32_t)a.cbits});
    return middle_phase_dispatch(a, lay, dst, FullGain{a.gain});
}

hipError_t launch_backward(const BackwardArgs &a)
{
    const hipStream_t st = a.stream;
    const bool separable = a.gain_kind == GAIN_LOG_SEPARABLE;
    const BackwardLayout lay = backward_layout(a.plan, a.K, a.B, int64_t(1) << a.cbits, separable);
    const uint64_t L = uint64_t(1) << a.K;
    hipError_t e = record(a.events[0], st);
    if (e != hipSuccess) return e;
    const bool want_dg = separable ? (a.dgt != nullptr) : (a.dgain != nullptr);
    // Both gradients with the three-pass plan: the fused path, whose first
    // launch covers 2*B*L/32 work-items (a 32-bit grid).
    if (want_dg && a.dx && a.B > 0 && a.plan == PLAN_THREE_PASS &&
        (uint64_t)a.B * L / 16u <= 0xffffffffull) {
        float *dst = separable ? a.ws + lay.dg : a.dgain;
        e = a.dtype == DTYPE_BF16 ? fused_gain<__bf16>(a, lay, dst) : fused_gain<float>(a, lay, dst);
        if (e != hipSuccess) return e;
        return record(a.events[2], st);
    }
    if (want_dg) {
        float *dst = separable ? a.ws + lay.dg : a.dgain;
        if (a.B == 0) {
            hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(L)), dim3(256), 0, st, dst, L);
            e = hipGetLastError();
        } else {
            e = a.dtype == DTYPE_BF16 ? grad_dispatch<__bf16>(a, lay, dst)
                                      : grad_dispatch<float>(a, lay, dst);
        }
        if (e != hipSuccess) return e;
        if (separable && (e = separable_reductions(a, lay, dst)) != hipSuccess)
            return e;
    }
    if ((e = record(a.events[1], st)) != hipSuccess) return e;
    if (a.dx && a.B > 0) {
        // dX = the mixer applied to dY, after dG so that dX may be dY itself
        LaunchArgs f{};
        f.x = a.dy;
        f.y = a.dx;
        f.gain_kind = a.gain_kind;
        f.gain = a.gain;
        f.gain_t = a.gain_t;
        f.gain_c = a.gain_c;
        f.cbits = a.cbits;
        f.ws = a.ws;
        f.B = a.B;
        f.K = a.K;
        f.nvalid = a.nvalid;
        f.dtype = a.dtype;
        f.plan = a.plan;
        f.stream = st;
        if ((e = launch(f)) != hipSuccess) return e;
    }
    return record(a.events[2], st);
}

}  // namespace whtmix
