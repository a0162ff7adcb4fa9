// Memory-system calibration for MI355X (gfx950), standalone program.
//
//   membw copy <MiB> <reps>   plain float4 copy of a buffer of <MiB>, <reps>
//                             launches (the reference for scaling rocprofv3
//                             FETCH_SIZE / WRITE_SIZE counters to bytes)
//   membw sweep               bandwidth characterisation:
//       copy    HBM copy rate, buffers rotated so nothing is cache resident
//       reread  one kernel re-reading a buffer many times: L2 (4 MiB per XCD)
//               and Infinity Cache residency as a function of size
//       pattern the WHTMix three-pass traffic (bf16 x -> f32 workspace ->
//               f32 workspace -> bf16 y, B=4 slices of 2^23) done by plain
//               copies: the floor for any three-pass schedule of that shape
//   membw fabric              traffic that leaves the XCDs (L2 misses), with
//                             eight 16-byte loads in flight per lane:
//       read    re-read of S bytes, the block -> data map rotated by one
//               block per launch so no XCD finds its data in its own L2:
//               Infinity Cache (S <= 256 MiB) vs HBM rate
//       wr+rd   write S bytes, then read them back (rotated)
//       rmw     in-place read-modify-write of a resident buffer
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>

#define CK(x)                                                                        \
    do {                                                                             \
        hipError_t e_ = (x);                                                         \
        if (e_ != hipSuccess) {                                                      \
            std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), \
                         __LINE__);                                                  \
            std::exit(1);                                                            \
        }                                                                            \
    } while (0)

namespace {

constexpr int kGrid = 2048, kBlock = 256;

__global__ void copy_f4(const float4 *__restrict__ in, float4 *__restrict__ out, size_t n4)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4; i += stride)
        out[i] = in[i];
}

__global__ void reread_f4(const float4 *__restrict__ in, float *__restrict__ sink, size_t n4,
                          int reps)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    float acc = 0.f;
    for (int r = 0; r < reps; ++r)
        for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4; i += stride) {
            const float4 v = in[i];
            acc += v.x + v.y + v.z + v.w;
        }
    sink[blockIdx.x * (size_t)blockDim.x + threadIdx.x] = acc;
}

// bf16 pairs -> float32 (exact widening), 4 elements per lane
__global__ void widen(const uint2 *__restrict__ in, float4 *__restrict__ out, size_t n4)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4; i += stride) {
        const uint2 u = in[i];
        out[i] = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                             __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
    }
}

__global__ void touch(float4 *__restrict__ s, size_t n4)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4; i += stride) {
        float4 v = s[i];
        v.x += 1.f;
        s[i] = v;
    }
}

// float32 -> bf16 by truncation (traffic stand-in only)
__global__ void narrow(const float4 *__restrict__ in, uint2 *__restrict__ out, size_t n4)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4; i += stride) {
        const float4 v = in[i];
        out[i] = make_uint2((__float_as_uint(v.x) >> 16) | (__float_as_uint(v.y) & 0xffff0000u),
                            (__float_as_uint(v.z) >> 16) | (__float_as_uint(v.w) & 0xffff0000u));
    }
}

// Chunks of BS*U float4 per block and iteration; chunk c is handled by block
// (c + rot) mod grid, so a rotation moves every chunk to another XCD.
constexpr int kU = 8, kBS = 256;

__device__ __forceinline__ size_t first_chunk(int rot)
{
    return (blockIdx.x + gridDim.x - (unsigned)rot % gridDim.x) % gridDim.x;
}

__global__ void __launch_bounds__(kBS)
fab_read(const float4 *__restrict__ in, float *__restrict__ sink, size_t n4, int rot)
{
    const size_t chunk = (size_t)kBS * kU, nch = n4 / chunk;
    float acc = 0.f;
    for (size_t c = first_chunk(rot); c < nch; c += gridDim.x) {
        float4 v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u)
            v[u] = in[c * chunk + u * kBS + threadIdx.x];
#pragma unroll
        for (int u = 0; u < kU; ++u)
            acc += v[u].x + v[u].y + v[u].z + v[u].w;
    }
    if (acc == 1234.5f)   // never true for the zero-filled buffers: keeps the loads
        sink[threadIdx.x] = acc;
}

__global__ void __launch_bounds__(kBS)
fab_write(float4 *__restrict__ out, size_t n4, int rot, float val)
{
    const size_t chunk = (size_t)kBS * kU, nch = n4 / chunk;
    for (size_t c = first_chunk(rot); c < nch; c += gridDim.x)
#pragma unroll
        for (int u = 0; u < kU; ++u)
            out[c * chunk + u * kBS + threadIdx.x] = make_float4(val, val, val, val);
}

__global__ void __launch_bounds__(kBS)
fab_rmw(float4 *__restrict__ s, size_t n4, int rot)
{
    const size_t chunk = (size_t)kBS * kU, nch = n4 / chunk;
    for (size_t c = first_chunk(rot); c < nch; c += gridDim.x) {
        float4 v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u)
            v[u] = s[c * chunk + u * kBS + threadIdx.x];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            v[u].x += 1.f;
            s[c * chunk + u * kBS + threadIdx.x] = v[u];
        }
    }
}

float elapsed(hipEvent_t a, hipEvent_t b)
{
    float ms = 0;
    CK(hipEventElapsedTime(&ms, a, b));
    return ms;
}

int do_copy(size_t mib, int reps)
{
    const size_t bytes = mib << 20;
    char *a, *b;
    CK(hipMalloc(&a, bytes));
    CK(hipMalloc(&b, bytes));
    CK(hipMemset(a, 0, bytes));
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    CK(hipEventRecord(e0, 0));
    for (int r = 0; r < reps; ++r)
        hipLaunchKernelGGL(copy_f4, dim3(kGrid), dim3(kBlock), 0, 0, (const float4 *)a,
                           (float4 *)b, bytes / 16);
    CK(hipGetLastError());
    CK(hipEventRecord(e1, 0));
    CK(hipEventSynchronize(e1));
    const float ms = elapsed(e0, e1);
    std::printf("copy %zu MiB x %d: %.1f us per launch, %.0f GB/s (read+write bytes %zu)\n", mib,
                reps, ms * 1e3 / reps, 2.0 * bytes * reps / (ms * 1e-3) / 1e9, 2 * bytes);
    CK(hipFree(a));
    CK(hipFree(b));
    return 0;
}

int do_sweep()
{
    const size_t MiB = 1 << 20;
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    float *sink;
    CK(hipMalloc(&sink, sizeof(float) * kGrid * kBlock));

    // HBM copy, rotating over 4 buffer pairs of 256 MiB (2 GiB footprint)
    {
        const size_t bytes = 256 * MiB;
        char *pool;
        CK(hipMalloc(&pool, 8 * bytes));
        CK(hipMemset(pool, 0, 8 * bytes));
        const int reps = 24;
        for (int r = 0; r < 4; ++r)
            hipLaunchKernelGGL(copy_f4, dim3(kGrid), dim3(kBlock), 0, 0,
                               (const float4 *)(pool + 2 * (r % 4) * bytes),
                               (float4 *)(pool + (2 * (r % 4) + 1) * bytes), bytes / 16);
        CK(hipDeviceSynchronize());
        CK(hipEventRecord(e0, 0));
        for (int r = 0; r < reps; ++r)
            hipLaunchKernelGGL(copy_f4, dim3(kGrid), dim3(kBlock), 0, 0,
                               (const float4 *)(pool + 2 * (r % 4) * bytes),
                               (float4 *)(pool + (2 * (r % 4) + 1) * bytes), bytes / 16);
        CK(hipEventRecord(e1, 0));
        CK(hipEventSynchronize(e1));
        std::printf("copy_hbm 256MiB_rotating %.0f GB/s\n",
                    2.0 * bytes * reps / (elapsed(e0, e1) * 1e-3) / 1e9);
        CK(hipFree(pool));
    }
    // steady-state re-read inside one kernel
    {
        char *buf;
        CK(hipMalloc(&buf, 512 * MiB));
        CK(hipMemset(buf, 0, 512 * MiB));
        const size_t sizes[] = {4, 8, 16, 32, 64, 128, 256, 512};
        for (size_t s : sizes) {
            const size_t n4 = s * MiB / 16;
            int reps = (int)(2048 / s);
            if (reps < 2) reps = 2;
            hipLaunchKernelGGL(reread_f4, dim3(kGrid), dim3(kBlock), 0, 0, (const float4 *)buf,
                               sink, n4, 1);
            CK(hipDeviceSynchronize());
            CK(hipEventRecord(e0, 0));
            hipLaunchKernelGGL(reread_f4, dim3(kGrid), dim3(kBlock), 0, 0, (const float4 *)buf,
                               sink, n4, reps);
            CK(hipEventRecord(e1, 0));
            CK(hipEventSynchronize(e1));
            std::printf("reread %zuMiB %.0f GB/s\n", s,
                        (double)s * MiB * reps / (elapsed(e0, e1) * 1e-3) / 1e9);
        }
        CK(hipFree(buf));
    }
    // three-pass traffic pattern by plain copies
    {
        const size_t L = (size_t)1 << 23, B = 4;
        const size_t xbytes = B * L * 2;
        const int nset = 5, steps = 50;
        char *X, *Y, *S;
        CK(hipMalloc(&X, nset * xbytes));
        CK(hipMalloc(&Y, nset * xbytes));
        CK(hipMalloc(&S, B * L * 4));
        CK(hipMemset(X, 0, nset * xbytes));
        CK(hipMemset(S, 0, B * L * 4));
        const size_t n4 = B * L / 4;
        auto step = [&](int it) {
            const uint2 *x = (const uint2 *)(X + (it % nset) * xbytes);
            uint2 *y = (uint2 *)(Y + (it % nset) * xbytes);
            hipLaunchKernelGGL(widen, dim3(kGrid), dim3(kBlock), 0, 0, x, (float4 *)S, n4);
            hipLaunchKernelGGL(touch, dim3(kGrid), dim3(kBlock), 0, 0, (float4 *)S, n4);
            hipLaunchKernelGGL(narrow, dim3(kGrid), dim3(kBlock), 0, 0, (const float4 *)S, y, n4);
        };
        for (int it = 0; it < 5; ++it) step(it);
        CK(hipDeviceSynchronize());
        CK(hipEventRecord(e0, 0));
        for (int it = 0; it < steps; ++it) step(it);
        CK(hipEventRecord(e1, 0));
        CK(hipEventSynchronize(e1));
        const double us = elapsed(e0, e1) * 1e3 / steps;
        const double bytes = (double)B * L * (2 + 4 + 4 + 4 + 4 + 2);
        std::printf("pattern three_pass_copies %.1f us per step, %.0f GB/s of moved bytes\n", us,
                    bytes / (us * 1e-6) / 1e9);
        CK(hipFree(X));
        CK(hipFree(Y));
        CK(hipFree(S));
    }
    CK(hipFree(sink));
    return 0;
}

int do_fabric()
{
    const size_t MiB = 1 << 20, total = 3072 * MiB;
    hipEvent_t e0, e1, e2;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    CK(hipEventCreate(&e2));
    float *sink;
    char *buf;
    CK(hipMalloc(&sink, sizeof(float) * kBS));
    CK(hipMalloc(&buf, total));
    CK(hipMemset(buf, 0, total));
    auto grid = [](size_t n4) {
        const size_t nch = n4 / ((size_t)kBS * kU);
        return (unsigned)(nch < (size_t)kGrid ? nch : (size_t)kGrid);
    };
    for (size_t s : {32, 64, 128, 192, 256, 512, 1024}) {
        const size_t n4 = s * MiB / 16;
        const int reps = 20;
        for (int r = 0; r < 3; ++r)
            hipLaunchKernelGGL(fab_read, dim3(grid(n4)), dim3(kBS), 0, 0, (const float4 *)buf, sink,
                               n4, r);
        CK(hipDeviceSynchronize());
        CK(hipEventRecord(e0, 0));
        for (int r = 0; r < reps; ++r)
            hipLaunchKernelGGL(fab_read, dim3(grid(n4)), dim3(kBS), 0, 0, (const float4 *)buf, sink,
                               n4, r + 3);
        CK(hipEventRecord(e1, 0));
        CK(hipEventSynchronize(e1));
        std::printf("read %zuMiB %.0f GB/s\n", s,
                    (double)s * MiB * reps / (elapsed(e0, e1) * 1e-3) / 1e9);
    }
    for (size_t s : {64, 128, 256, 512}) {
        const size_t n4 = s * MiB / 16;
        const int reps = 10;
        double tw = 0, tr = 0;
        for (int r = 0; r < reps + 2; ++r) {
            // evict: read 2 GiB elsewhere
            hipLaunchKernelGGL(fab_read, dim3(kGrid), dim3(kBS), 0, 0,
                               (const float4 *)(buf + 1024 * MiB), sink, 2048 * MiB / 16, 0);
            CK(hipEventRecord(e0, 0));
            hipLaunchKernelGGL(fab_write, dim3(grid(n4)), dim3(kBS), 0, 0, (float4 *)buf, n4, r,
                               0.0f);
            CK(hipEventRecord(e1, 0));
            hipLaunchKernelGGL(fab_read, dim3(grid(n4)), dim3(kBS), 0, 0, (const float4 *)buf, sink,
                               n4, r + 1);
            CK(hipEventRecord(e2, 0));
            CK(hipEventSynchronize(e2));
            if (r >= 2) {
                tw += elapsed(e0, e1);
                tr += elapsed(e1, e2);
            }
        }
        std::printf("wr+rd %zuMiB write %.0f GB/s read %.0f GB/s\n", s,
                    (double)s * MiB * reps / (tw * 1e-3) / 1e9,
                    (double)s * MiB * reps / (tr * 1e-3) / 1e9);
    }
    for (size_t s : {64, 128}) {
        const size_t n4 = s * MiB / 16;
        const int reps = 20;
        for (int r = 0; r < 3; ++r)
            hipLaunchKernelGGL(fab_rmw, dim3(grid(n4)), dim3(kBS), 0, 0, (float4 *)buf, n4, r);
        CK(hipDeviceSynchronize());
        CK(hipEventRecord(e0, 0));
        for (int r = 0; r < reps; ++r)
            hipLaunchKernelGGL(fab_rmw, dim3(grid(n4)), dim3(kBS), 0, 0, (float4 *)buf, n4, r + 3);
        CK(hipEventRecord(e1, 0));
        CK(hipEventSynchronize(e1));
        std::printf("rmw %zuMiB %.0f GB/s (read + written bytes)\n", s,
                    2.0 * s * MiB * reps / (elapsed(e0, e1) * 1e-3) / 1e9);
    }
    CK(hipGetLastError());
    CK(hipFree(buf));
    CK(hipFree(sink));
    return 0;
}

}  // namespace

int main(int argc, char **argv)
{
    if (argc >= 2 && std::strcmp(argv[1], "copy") == 0) {
        const size_t mib = argc >= 3 ? std::strtoul(argv[2], nullptr, 10) : 256;
        const int reps = argc >= 4 ? std::atoi(argv[3]) : 10;
        if (mib < 1 || mib > 8192 || reps < 1 || reps > 10000) {
            std::fprintf(stderr, "copy size must be 1..8192 MiB, reps 1..10000\n");
            return 2;
        }
        return do_copy(mib, reps);
    }
    if (argc >= 2 && std::strcmp(argv[1], "sweep") == 0)
        return do_sweep();
    if (argc >= 2 && std::strcmp(argv[1], "fabric") == 0)
        return do_fabric();
    std::fprintf(stderr, "usage: membw copy <MiB> <reps> | membw sweep | membw fabric\n");
    return 2;
}
