// C entry points of the WHTMix library: argument checks, plan choice,
// per-(device, stream) workspace, status text.  Declared in include/whtmix.h.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>

#include "whtmix.h"
#include "whtmix_launch.h"
#include "whtmix_module.h"
#include "whtmix_plan.h"

namespace {

thread_local std::string g_last_error;

struct Workspace {
    float *ptr = nullptr;
    int64_t bytes = 0;
    // ONE_LAUNCH counter block (kCounterWords words), allocated and zeroed
    // once; each call's kernel returns it to zero (the sticky error word
    // aside, which whtmix_stream_status reads and clears).
    uint32_t *ctr = nullptr;
};

// Keyed by (device, stream).  The mutex is held from workspace lookup until
// the kernels that use the workspace are enqueued, so a concurrent call that
// grows (frees and reallocates) the same stream's workspace cannot free it
// between lookup and launch.
std::mutex g_ws_mutex;
std::map<std::pair<int, void *>, Workspace> g_ws;

bool is_pow2(int64_t v) { return v >= 1 && (v & (v - 1)) == 0; }

int log2_exact(int64_t v)
{
    int k = 0;
    while ((int64_t(1) << k) < v) ++k;
    return k;
}

bool overlaps(uintptr_t a, uint64_t na, uintptr_t b, uint64_t nb)
{
    return a < b + nb && b < a + na;
}

struct Checked {
    int K = 0;
    int64_t n_pad = 0;
    int plan = whtmix::PLAN_AUTO;
    int kernels = 0;
    whtmix::Split split{0, 0, 0};
    int64_t ws_bytes = 0;
    int elt = 4;
};

// Shape, dtype and option checks shared by forward and describe.
int check_shape(int64_t B, int64_t N, int64_t C, int dtype, const whtmix_options *opt,
                Checked *out)
{
    if (dtype != WHTMIX_DTYPE_F32 && dtype != WHTMIX_DTYPE_BF16)
        return WHTMIX_ERROR_UNSUPPORTED_DTYPE;
    if (B < 0 || N < 1)
        return WHTMIX_ERROR_INVALID_VALUE;
    if (!is_pow2(C))
        return WHTMIX_ERROR_NOT_POWER_OF_TWO;
    if (N > (int64_t(1) << whtmix::kMaxLog2Slice))
        return WHTMIX_ERROR_TOO_LARGE;
    // Rows N .. N_pad-1 count as zeros so that H_N acts on a power-of-two
    // length (section III-B).
    const int nbits = log2_exact(N);
    const int K = nbits + log2_exact(C);
    if (K > whtmix::kMaxLog2Slice)
        return WHTMIX_ERROR_TOO_LARGE;
    const int64_t L = int64_t(1) << K;
    // Work-items per launch are B*L/32 (tiled plans) or B*256 (small plan);
    // both must stay below 2^32 (the grid size is a 32-bit count).
    if (B > ((int64_t(1) << 37) - 1) / L)
        return WHTMIX_ERROR_TOO_LARGE;
    if (K <= whtmix::kMaxSmall && B >= (int64_t(1) << 24))
        return WHTMIX_ERROR_TOO_LARGE;
    int plan = opt ? opt->plan : whtmix::PLAN_AUTO;
    // The wave-tile plans move x and y in 16-byte groups of up to 8 elements.
    const bool wave_ok = K >= whtmix::kWaveMinK && K <= whtmix::kWaveMaxK && (N * C) % 8 == 0;
    switch (plan) {
    case whtmix::PLAN_AUTO:
        plan = K <= whtmix::kMaxSmall ? whtmix::PLAN_SMALL
               : K == whtmix::kMaxTile && wave_ok && B <= whtmix::kTwoPass15MaxBatch
                   ? whtmix::PLAN_TWO_PASS
               : K <= whtmix::kMaxTile ? whtmix::PLAN_FUSED
               : K == whtmix::kMaxFused && B >= whtmix::kFusedPairMinBatch ? whtmix::PLAN_FUSED
               : K == whtmix::kMaxFused && wave_ok && B <= whtmix::kWave16MaxBatch
                   ? whtmix::PLAN_WAVE_TILES
               : K == whtmix::kMaxFused && wave_ok && B <= whtmix::kTwoPass16MaxBatch
                   ? whtmix::PLAN_TWO_PASS
                   : whtmix::PLAN_THREE_PASS;
        break;
    case whtmix::PLAN_WAVE_TILES:
        if (!wave_ok) return WHTMIX_ERROR_INVALID_VALUE;
        // one 64-thread workgroup per 2^9 elements: B*L/8 work-items
        if (B > ((int64_t(1) << 35) - 1) / L) return WHTMIX_ERROR_TOO_LARGE;
        break;
    case whtmix::PLAN_TWO_PASS:
        if (!wave_ok || K < whtmix::kTwoPassMinK) return WHTMIX_ERROR_INVALID_VALUE;
        // the fold pass runs B*L/8 work-items with B rounded up to a multiple of 8
        if ((B + 7) / 8 * 8 > ((int64_t(1) << 35) - 1) / L) return WHTMIX_ERROR_TOO_LARGE;
        break;
    case whtmix::PLAN_ONE_LAUNCH:
        if (!wave_ok || B > whtmix::kOneLaunchMaxBatch) return WHTMIX_ERROR_INVALID_VALUE;
        break;
    case whtmix::PLAN_SMALL:
        if (K > whtmix::kMaxSmall) return WHTMIX_ERROR_INVALID_VALUE;
        break;
    case whtmix::PLAN_FUSED:
        if (K < whtmix::kMinTile || K > whtmix::kMaxFused) return WHTMIX_ERROR_INVALID_VALUE;
        break;
    case whtmix::PLAN_THREE_PASS:
        if (K < whtmix::kMinTile + 1) return WHTMIX_ERROR_INVALID_VALUE;
        break;
    default:
        return WHTMIX_ERROR_INVALID_VALUE;
    }
    out->K = K;
    out->n_pad = int64_t(1) << nbits;
    out->plan = plan;
    out->elt = dtype == WHTMIX_DTYPE_BF16 ? 2 : 4;
    out->kernels = plan == whtmix::PLAN_THREE_PASS || plan == whtmix::PLAN_WAVE_TILES ? 3
                   : plan == whtmix::PLAN_TWO_PASS                                  ? 2
                                                                                    : 1;
    if (plan == whtmix::PLAN_THREE_PASS) {
        out->split = whtmix::three_pass_split(K);
        out->ws_bytes = B * L * 4;
    }
    if (plan == whtmix::PLAN_WAVE_TILES || plan == whtmix::PLAN_ONE_LAUNCH ||
        plan == whtmix::PLAN_TWO_PASS) {
        out->split = whtmix::Split{9, K - 9, 18 - K};
        out->ws_bytes = B * L * 4;
    }
    return WHTMIX_SUCCESS;
}

// The plan the backward pass and the block take for a forward plan.  The
// single-workgroup FUSED plan reaches 2^16 elements (two register sets) and
// the wave-tile plans exist in the mixer's forward only: the backward pass
// and the block run slices of 2^16 with the three-pass plan, and the
// wave-tile plans' smaller slices with FUSED (THREE_PASS when forced to
// ONE_LAUNCH).
void three_pass_beyond_one_tile(int64_t B, Checked *c)
{
    if ((c->plan == whtmix::PLAN_WAVE_TILES || c->plan == whtmix::PLAN_TWO_PASS) &&
        c->K <= whtmix::kMaxTile) {
        c->plan = whtmix::PLAN_FUSED;
        c->kernels = 1;
        c->split = whtmix::Split{0, 0, 0};
        c->ws_bytes = 0;
        return;
    }
    if ((c->plan == whtmix::PLAN_FUSED && c->K > whtmix::kMaxTile) ||
        c->plan == whtmix::PLAN_ONE_LAUNCH || c->plan == whtmix::PLAN_WAVE_TILES ||
        c->plan == whtmix::PLAN_TWO_PASS) {
        c->plan = whtmix::PLAN_THREE_PASS;
        c->kernels = 3;
        c->split = whtmix::three_pass_split(c->K);
        c->ws_bytes = B * (int64_t(1) << c->K) * 4;
    }
}

int hip_fail(hipError_t e, const char *what)
{
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return e == hipErrorOutOfMemory ? WHTMIX_ERROR_OUT_OF_MEMORY : WHTMIX_ERROR_HIP;
}

// Returns a workspace of at least `bytes` for (current device, stream).
// Caller holds g_ws_mutex.
int get_workspace(void *stream, int64_t bytes, float **out)
{
    // Test hook: with WHTMIX_TEST_FAIL_WORKSPACE set in the environment every
    // workspace request fails as an allocation failure would, before any HIP
    // call, so the status path can be tested without exhausting the device.
    if (std::getenv("WHTMIX_TEST_FAIL_WORKSPACE")) {
        g_last_error = "workspace allocation refused (WHTMIX_TEST_FAIL_WORKSPACE)";
        return WHTMIX_ERROR_OUT_OF_MEMORY;
    }
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    Workspace &w = g_ws[{dev, stream}];
    if (w.bytes < bytes) {
        if (w.ptr) {
            // Work already enqueued on this stream may still read the old
            // buffer; let it finish before freeing.
            e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
            if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
            e = hipFree(w.ptr);
            w.ptr = nullptr;
            w.bytes = 0;
            if (e != hipSuccess) return hip_fail(e, "hipFree");
        }
        void *p = nullptr;
        e = hipMalloc(&p, (size_t)bytes);
        if (e != hipSuccess) {
            g_last_error = std::string("hipMalloc of workspace (") + std::to_string(bytes) +
                           " bytes): " + hipGetErrorString(e);
            (void)hipGetLastError();
            return WHTMIX_ERROR_OUT_OF_MEMORY;
        }
        w.ptr = static_cast<float *>(p);
        w.bytes = bytes;
    }
    *out = w.ptr;
    return WHTMIX_SUCCESS;
}

// The ONE_LAUNCH counter block of (current device, stream), allocated and
// zeroed on first use.  Caller holds g_ws_mutex.
int get_counters(void *stream, uint32_t **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    Workspace &w = g_ws[{dev, stream}];
    if (!w.ctr) {
        void *p = nullptr;
        const size_t bytes = sizeof(uint32_t) * whtmix::kCounterWords;
        e = hipMalloc(&p, bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            g_last_error = std::string("hipMalloc of counters: ") + hipGetErrorString(e);
            return WHTMIX_ERROR_OUT_OF_MEMORY;
        }
        e = hipMemset(p, 0, bytes);
        if (e != hipSuccess) {
            (void)hipFree(p);
            return hip_fail(e, "hipMemset of counters");
        }
        w.ctr = static_cast<uint32_t *>(p);
    }
    *out = w.ctr;
    return WHTMIX_SUCCESS;
}

}  // namespace

extern "C" {

int whtmix_plan_describe(int64_t B, int64_t N, int64_t C, int dtype,
                         const whtmix_options *options, whtmix_plan_info *info)
{
    if (!info) return WHTMIX_ERROR_INVALID_VALUE;
    Checked c;
    int st = check_shape(B, N, C, dtype, options, &c);
    if (st != WHTMIX_SUCCESS) return st;
    info->plan = c.plan;
    info->kernels = c.kernels;
    info->log2_slice = c.K;
    const bool passes = c.plan == whtmix::PLAN_THREE_PASS || c.plan == whtmix::PLAN_ONE_LAUNCH ||
                        c.plan == whtmix::PLAN_WAVE_TILES || c.plan == whtmix::PLAN_TWO_PASS;
    info->outer_bits = passes ? c.split.A : 0;
    info->run_bits = passes ? c.split.R : 0;
    info->workspace_bytes = c.ws_bytes;
    info->padded_tokens = c.n_pad;
    const int cbits = log2_exact(C);
    Checked blk = c;   // the block's plan
    three_pass_beyond_one_tile(B, &blk);
    info->module_path = cbits <= whtmix::kModuleMaxCbits
                            ? whtmix::module_path(blk.plan, cbits, dtype, blk.K)
                            : -1;
    info->module_outer_bits =
        info->module_path >= 0 && blk.plan == whtmix::PLAN_THREE_PASS
            ? whtmix::module_outer_bits(info->module_path, cbits, blk.K)
            : 0;
    info->module_backward_fused =
        whtmix::module_backward_fused(blk.plan, cbits, dtype, blk.K) ? 1 : 0;
    return WHTMIX_SUCCESS;
}

}  // extern "C"

namespace {

// noalloc: the three-pass, two-pass or wave-tile workspace is the fixed device scratch
// instead of the per-stream workspace, and nothing is allocated.
int forward_impl(const void *x, int gain_kind, const float *gain, const float *gain_t,
                 const float *gain_c, void *y, int64_t B, int64_t N, int64_t C, int dtype,
                 void *stream, const whtmix_options *options, bool noalloc = false)
{
    Checked c;
    int st = check_shape(B, N, C, dtype, options, &c);
    if (st != WHTMIX_SUCCESS) return st;
    if (B == 0) return WHTMIX_SUCCESS;
    const bool full = gain_kind == whtmix::GAIN_FULL;
    if (!x || !y || (full ? !gain : (!gain_t || !gain_c))) return WHTMIX_ERROR_INVALID_VALUE;
    const uintptr_t px = reinterpret_cast<uintptr_t>(x);
    const uintptr_t py = reinterpret_cast<uintptr_t>(y);
    const uintptr_t pg = reinterpret_cast<uintptr_t>(full ? gain : gain_t);
    const uintptr_t pc = reinterpret_cast<uintptr_t>(full ? gain : gain_c);
    if ((px | py | pg | pc) & 15u) return WHTMIX_ERROR_MISALIGNED;
    const uint64_t xy_bytes = (uint64_t)B * (uint64_t)N * (uint64_t)C * (uint64_t)c.elt;
    if (px != py && overlaps(px, xy_bytes, py, xy_bytes)) return WHTMIX_ERROR_INVALID_VALUE;
    if (full) {
        if (overlaps(pg, (uint64_t)c.n_pad * C * 4, py, xy_bytes))
            return WHTMIX_ERROR_INVALID_VALUE;
    } else if (overlaps(pg, (uint64_t)c.n_pad * 4, py, xy_bytes) ||
               overlaps(pc, (uint64_t)C * 4, py, xy_bytes)) {
        return WHTMIX_ERROR_INVALID_VALUE;
    }

    whtmix::LaunchArgs a{};
    a.x = x;
    a.y = y;
    a.gain_kind = gain_kind;
    a.gain = gain;
    a.gain_t = gain_t;
    a.gain_c = gain_c;
    a.cbits = log2_exact(C);
    a.B = B;
    a.K = c.K;
    a.nvalid = (uint32_t)(N * C);
    a.dtype = dtype;
    a.plan = c.plan;
    a.stream = static_cast<hipStream_t>(stream);
    for (int i = 0; i < 4; ++i)
        a.events[i] = options ? static_cast<hipEvent_t>(options->events[i]) : nullptr;

    const bool wave = c.plan == whtmix::PLAN_WAVE_TILES || c.plan == whtmix::PLAN_ONE_LAUNCH ||
                      c.plan == whtmix::PLAN_TWO_PASS;
    const bool uses_ws = c.plan == whtmix::PLAN_THREE_PASS || c.plan == whtmix::PLAN_WAVE_TILES ||
                         c.plan == whtmix::PLAN_TWO_PASS;
    if (noalloc && uses_ws) {
        if (c.ws_bytes > whtmix::kNoAllocScratchFloats * 4) {
            g_last_error = "whtmix_forward_noalloc: the call needs " + std::to_string(c.ws_bytes) +
                           " bytes of workspace, more than the fixed " +
                           std::to_string(whtmix::kNoAllocScratchFloats * 4) +
                           "-byte scratch (B * N_pad * C <= 2^23)";
            return WHTMIX_ERROR_TOO_LARGE;
        }
        hipError_t e = whtmix::noalloc_scratch(&a.ws);
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress of the scratch");
        e = wave ? whtmix::launch_wave(a) : whtmix::launch(a);
        if (e != hipSuccess) return hip_fail(e, "kernel launch");
        return WHTMIX_SUCCESS;
    }
    if (uses_ws) {
        std::lock_guard<std::mutex> lock(g_ws_mutex);
        st = get_workspace(stream, c.ws_bytes, &a.ws);
        if (st != WHTMIX_SUCCESS) return st;
        hipError_t e = wave ? whtmix::launch_wave(a) : whtmix::launch(a);
        if (e != hipSuccess) return hip_fail(e, "kernel launch");
        return WHTMIX_SUCCESS;
    }
    if (c.plan == whtmix::PLAN_ONE_LAUNCH) {
        a.spin_limit = options && options->spin_limit ? options->spin_limit
                                                       : whtmix::kDefaultSpinLimit;
        std::lock_guard<std::mutex> lock(g_ws_mutex);
        st = get_workspace(stream, c.ws_bytes, &a.ws);
        if (st != WHTMIX_SUCCESS) return st;
        st = get_counters(stream, &a.counters);
        if (st != WHTMIX_SUCCESS) return st;
        hipError_t e = whtmix::launch_wave(a);
        if (e != hipSuccess) return hip_fail(e, "kernel launch");
        return WHTMIX_SUCCESS;
    }
    hipError_t e = whtmix::launch(a);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return WHTMIX_SUCCESS;
}

}  // namespace

extern "C" {

int whtmix_forward_ex(const void *x, const float *gain, void *y, int64_t B, int64_t N,
                      int64_t C, int dtype, void *stream, const whtmix_options *options)
{
    return forward_impl(x, whtmix::GAIN_FULL, gain, nullptr, nullptr, y, B, N, C, dtype, stream,
                        options);
}

int whtmix_forward_separable(const void *x, const float *log_gain_tokens,
                             const float *log_gain_channels, void *y, int64_t B, int64_t N,
                             int64_t C, int dtype, void *stream, const whtmix_options *options)
{
    return forward_impl(x, whtmix::GAIN_LOG_SEPARABLE, nullptr, log_gain_tokens,
                        log_gain_channels, y, B, N, C, dtype, stream, options);
}

}  // extern "C"

namespace {

struct Span {
    uintptr_t p;
    uint64_t n;
};

bool spans_overlap(Span a, Span b) { return a.p && b.p && overlaps(a.p, a.n, b.p, b.n); }

int backward_impl(const void *x, const void *dy, int gain_kind, const float *gain,
                  const float *gain_t, const float *gain_c, void *dx, float *dgain, float *dgt,
                  float *dgc, int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                  const whtmix_options *options)
{
    Checked c;
    int st = check_shape(B, N, C, dtype, options, &c);
    if (st != WHTMIX_SUCCESS) return st;
    three_pass_beyond_one_tile(B, &c);
    const bool sep = gain_kind == whtmix::GAIN_LOG_SEPARABLE;
    const bool want_dg = sep ? (dgt != nullptr || dgc != nullptr) : dgain != nullptr;
    if (sep && (dgt == nullptr) != (dgc == nullptr)) return WHTMIX_ERROR_INVALID_VALUE;
    if (!want_dg && !dx) return WHTMIX_ERROR_INVALID_VALUE;
    if (sep ? (!gain_t || !gain_c) : !gain) return WHTMIX_ERROR_INVALID_VALUE;
    if (B > 0 && (!dy || (want_dg && !x))) return WHTMIX_ERROR_INVALID_VALUE;
    const uint64_t xy = (uint64_t)B * (uint64_t)N * (uint64_t)C * (uint64_t)c.elt;
    const uint64_t P = (uint64_t)c.n_pad;
    Span sx{B > 0 && want_dg ? reinterpret_cast<uintptr_t>(x) : 0, xy};
    Span sdy{B > 0 ? reinterpret_cast<uintptr_t>(dy) : 0, xy};
    Span sdx{B > 0 ? reinterpret_cast<uintptr_t>(dx) : 0, xy};
    Span sg{reinterpret_cast<uintptr_t>(sep ? gain_t : gain), sep ? P * 4 : P * C * 4};
    Span sgc{reinterpret_cast<uintptr_t>(sep ? gain_c : nullptr), (uint64_t)C * 4};
    Span sdg{reinterpret_cast<uintptr_t>(dgain), P * C * 4};
    Span sdgt{reinterpret_cast<uintptr_t>(dgt), P * 4};
    Span sdgc{reinterpret_cast<uintptr_t>(dgc), (uint64_t)C * 4};
    const Span inputs[] = {sx, sdy, sg, sgc};
    const Span outputs[] = {sdx, sdg, sdgt, sdgc};
    for (const Span &s : inputs)
        if (s.p & 15u) return WHTMIX_ERROR_MISALIGNED;
    for (const Span &s : outputs)
        if (s.p & 15u) return WHTMIX_ERROR_MISALIGNED;
    // No output may overlap an input or another output, except that dx may
    // be dy itself (the gain gradient is computed before dx is written).
    for (int i = 0; i < 4; ++i) {
        const Span &o = outputs[i];
        if (!o.p) continue;
        for (int j = 0; j < 4; ++j) {
            if (i == 0 && j == 1 && o.p == inputs[j].p) continue;
            if (spans_overlap(o, inputs[j])) return WHTMIX_ERROR_INVALID_VALUE;
        }
        for (int j = 0; j < 4; ++j)
            if (j != i && spans_overlap(o, outputs[j])) return WHTMIX_ERROR_INVALID_VALUE;
    }
    if (B == 0 && !want_dg) return WHTMIX_SUCCESS;

    whtmix::BackwardArgs a{};
    a.x = x;
    a.dy = dy;
    a.dx = B > 0 ? dx : nullptr;
    a.gain_kind = gain_kind;
    a.gain = gain;
    a.gain_t = gain_t;
    a.gain_c = gain_c;
    a.dgain = dgain;
    a.dgt = dgt;
    a.dgc = dgc;
    a.cbits = log2_exact(C);
    a.B = B;
    a.K = c.K;
    a.nvalid = (uint32_t)(N * C);
    a.dtype = dtype;
    a.plan = c.plan;
    a.stream = static_cast<hipStream_t>(stream);
    for (int i = 0; i < 4; ++i)
        a.events[i] = options ? static_cast<hipEvent_t>(options->events[i]) : nullptr;
    const whtmix::BackwardLayout lay = whtmix::backward_layout(c.plan, c.K, B, C, sep);
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    if (lay.floats > 0) {
        st = get_workspace(stream, (int64_t)(lay.floats * 4), &a.ws);
        if (st != WHTMIX_SUCCESS) return st;
    }
    hipError_t e = whtmix::launch_backward(a);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return WHTMIX_SUCCESS;
}

int module_impl(const void *x, const void *w_in, int gain_kind, const float *gain,
                const float *gain_t, const float *gain_c, const void *w_out, void *y, int64_t B,
                int64_t N, int64_t C, int dtype, void *stream, const whtmix_options *options)
{
    Checked c;
    int st = check_shape(B, N, C, dtype, options, &c);
    if (st != WHTMIX_SUCCESS) return st;
    three_pass_beyond_one_tile(B, &c);
    const int cbits = log2_exact(C);
    if (cbits > whtmix::kModuleMaxCbits) return WHTMIX_ERROR_TOO_LARGE;
    if (B == 0) return WHTMIX_SUCCESS;
    const bool full = gain_kind == whtmix::GAIN_FULL;
    if (!x || !y || !w_in || !w_out || (full ? !gain : (!gain_t || !gain_c)))
        return WHTMIX_ERROR_INVALID_VALUE;
    const uint64_t xy = (uint64_t)B * (uint64_t)N * (uint64_t)C * (uint64_t)c.elt;
    const uint64_t wb = (uint64_t)C * (uint64_t)C * (uint64_t)c.elt;
    const uint64_t P = (uint64_t)c.n_pad;
    const Span sy{reinterpret_cast<uintptr_t>(y), xy};
    const Span inputs[] = {{reinterpret_cast<uintptr_t>(x), xy},
                           {reinterpret_cast<uintptr_t>(w_in), wb},
                           {reinterpret_cast<uintptr_t>(w_out), wb},
                           {reinterpret_cast<uintptr_t>(full ? gain : gain_t),
                            full ? P * (uint64_t)C * 4 : P * 4},
                           {reinterpret_cast<uintptr_t>(full ? nullptr : gain_c),
                            (uint64_t)C * 4}};
    if (sy.p & 15u) return WHTMIX_ERROR_MISALIGNED;
    for (const Span &s : inputs)
        if (s.p & 15u) return WHTMIX_ERROR_MISALIGNED;
    // y may be x itself; no other overlap with an input.
    for (int i = 0; i < 5; ++i) {
        if (i == 0 && inputs[i].p == sy.p) continue;
        if (spans_overlap(sy, inputs[i])) return WHTMIX_ERROR_INVALID_VALUE;
    }

    whtmix::ModuleArgs m{};
    m.x = x;
    m.w_in = w_in;
    m.w_out = w_out;
    m.y = y;
    m.gain_kind = gain_kind;
    m.gain = gain;
    m.gain_t = gain_t;
    m.gain_c = gain_c;
    m.cbits = cbits;
    m.B = B;
    m.K = c.K;
    m.nvalid = (uint32_t)(N * C);
    m.dtype = dtype;
    m.plan = c.plan;
    m.stream = static_cast<hipStream_t>(stream);
    for (int i = 0; i < 4; ++i)
        m.events[i] = options ? static_cast<hipEvent_t>(options->events[i]) : nullptr;
    const int path = whtmix::module_path(c.plan, cbits, dtype, c.K);
    // workspace: mixer (THREE_PASS), then packed weights or Z, 256-byte aligned
    const int64_t mix = path == whtmix::MODULE_SMALL ? 0 : c.ws_bytes;
    // FUSED_MFMA: the packed weights; UNFUSED: Z, then the packed weights
    const int64_t zbytes = path == whtmix::MODULE_UNFUSED ? (B * N * C * 4 + 255) / 256 * 256 : 0;
    const int64_t extra = path == whtmix::MODULE_SMALL ? 0 : zbytes + (int64_t)(2 * wb);
    const int64_t off = (mix + 255) / 256 * 256;
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    float *ws = nullptr;
    if (off + extra > 0) {
        st = get_workspace(stream, off + extra, &ws);
        if (st != WHTMIX_SUCCESS) return st;
    }
    m.ws = mix > 0 ? ws : nullptr;
    void *tail = ws ? static_cast<void *>(reinterpret_cast<char *>(ws) + off) : nullptr;
    if (path == whtmix::MODULE_FUSED_MFMA) m.wpack = tail;
    if (path == whtmix::MODULE_UNFUSED) {
        m.z = static_cast<float *>(tail);
        m.wpack = static_cast<char *>(tail) + zbytes;
    }
    hipError_t e = whtmix::launch_module(m);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return WHTMIX_SUCCESS;
}

int64_t align256(int64_t v) { return (v + 255) / 256 * 256; }

int module_backward_impl(const void *x, const void *w_in, int gain_kind, const float *gain,
                         const float *gain_t, const float *gain_c, const void *w_out,
                         const void *dy, void *dx, float *dw_in, float *dw_out, float *dgain,
                         float *dgt, float *dgc, int64_t B, int64_t N, int64_t C, int dtype,
                         void *stream, const whtmix_options *options)
{
    Checked c;
    int st = check_shape(B, N, C, dtype, options, &c);
    if (st != WHTMIX_SUCCESS) return st;
    three_pass_beyond_one_tile(B, &c);
    const int cbits = log2_exact(C);
    if (cbits > whtmix::kModuleMaxCbits || B * N >= (int64_t(1) << 31))
        return WHTMIX_ERROR_TOO_LARGE;
    const bool sep = gain_kind == whtmix::GAIN_LOG_SEPARABLE;
    if (!w_in || !w_out || !dw_in || !dw_out || (sep ? (!gain_t || !gain_c) : !gain))
        return WHTMIX_ERROR_INVALID_VALUE;
    if (sep && (dgt == nullptr) != (dgc == nullptr)) return WHTMIX_ERROR_INVALID_VALUE;
    if (B > 0 && (!x || !dy || !dx)) return WHTMIX_ERROR_INVALID_VALUE;
    const uint64_t xy = (uint64_t)B * (uint64_t)N * (uint64_t)C * (uint64_t)c.elt;
    const uint64_t wb = (uint64_t)C * (uint64_t)C * (uint64_t)c.elt;
    const uint64_t P = (uint64_t)c.n_pad;
    const Span inputs[] = {{B > 0 ? reinterpret_cast<uintptr_t>(x) : 0, xy},
                           {B > 0 ? reinterpret_cast<uintptr_t>(dy) : 0, xy},
                           {reinterpret_cast<uintptr_t>(w_in), wb},
                           {reinterpret_cast<uintptr_t>(w_out), wb},
                           {reinterpret_cast<uintptr_t>(sep ? gain_t : gain),
                            sep ? P * 4 : P * (uint64_t)C * 4},
                           {reinterpret_cast<uintptr_t>(sep ? gain_c : nullptr), (uint64_t)C * 4}};
    const Span outputs[] = {{B > 0 ? reinterpret_cast<uintptr_t>(dx) : 0, xy},
                            {reinterpret_cast<uintptr_t>(dw_in), (uint64_t)C * C * 4},
                            {reinterpret_cast<uintptr_t>(dw_out), (uint64_t)C * C * 4},
                            {reinterpret_cast<uintptr_t>(dgain), P * (uint64_t)C * 4},
                            {reinterpret_cast<uintptr_t>(dgt), P * 4},
                            {reinterpret_cast<uintptr_t>(dgc), (uint64_t)C * 4}};
    for (const Span &s : inputs)
        if (s.p & 15u) return WHTMIX_ERROR_MISALIGNED;
    for (const Span &s : outputs)
        if (s.p & 15u) return WHTMIX_ERROR_MISALIGNED;
    // No output may overlap an input or another output, except dx == dy: dY
    // is consumed before dX is written (x is read after it).
    for (int i = 0; i < 6; ++i) {
        const Span &o = outputs[i];
        if (!o.p) continue;
        for (int j = 0; j < 6; ++j) {
            if (i == 0 && j == 1 && o.p == inputs[j].p) continue;
            if (spans_overlap(o, inputs[j])) return WHTMIX_ERROR_INVALID_VALUE;
        }
        for (int j = 0; j < 6; ++j)
            if (j != i && spans_overlap(o, outputs[j])) return WHTMIX_ERROR_INVALID_VALUE;
    }

    whtmix::ModuleBackwardArgs m{};
    m.x = x;
    m.w_in = w_in;
    m.w_out = w_out;
    m.dy = dy;
    m.dx = dx;
    m.dw_in = dw_in;
    m.dw_out = dw_out;
    m.gain_kind = gain_kind;
    m.gain = gain;
    m.gain_t = gain_t;
    m.gain_c = gain_c;
    m.dgain = dgain;
    m.dgt = dgt;
    m.dgc = dgc;
    m.cbits = cbits;
    m.B = B;
    m.K = c.K;
    m.nvalid = (uint32_t)(N * C);
    m.dtype = dtype;
    m.plan = c.plan;
    m.stream = static_cast<hipStream_t>(stream);
    for (int i = 0; i < 4; ++i)
        m.events[i] = options ? static_cast<hipEvent_t>(options->events[i]) : nullptr;
    // workspace: Z, Z', dZ'; packed weights; weight-gradient partials; the
    // mixer's forward and backward workspaces
    const int64_t rows = B * N;
    const int64_t zb = align256(rows * C * 4);
    const int64_t pk = align256((int64_t)(3 * wb));
    const whtmix::WgradPlan wp = whtmix::wgrad_plan((uint64_t)rows, cbits);
    const int64_t part = align256((int64_t)wp.partial_floats(cbits) * 4);
    const int64_t mix = align256(c.ws_bytes);
    const whtmix::BackwardLayout lay = whtmix::backward_layout(c.plan, c.K, B, C, sep);
    const int64_t bwd = align256((int64_t)(lay.floats * 4));
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    float *ws = nullptr;
    st = get_workspace(stream, 3 * zb + pk + part + mix + bwd, &ws);
    if (st != WHTMIX_SUCCESS) return st;
    char *p = reinterpret_cast<char *>(ws);
    m.z = reinterpret_cast<float *>(p);
    m.zp = reinterpret_cast<float *>(p + zb);
    m.dzp = reinterpret_cast<float *>(p + 2 * zb);
    m.wpack = p + 3 * zb;
    m.wpart = reinterpret_cast<float *>(p + 3 * zb + pk);
    m.mix_ws = mix > 0 ? reinterpret_cast<float *>(p + 3 * zb + pk + part) : nullptr;
    m.bwd_ws = bwd > 0 ? reinterpret_cast<float *>(p + 3 * zb + pk + part + mix) : nullptr;
    hipError_t e = whtmix::launch_module_backward(m);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return WHTMIX_SUCCESS;
}

}  // namespace

extern "C" {

int whtmix_module_backward(const void *x, const void *w_in, const float *gain, const void *w_out,
                           const void *dy, void *dx, float *dw_in, float *dw_out, float *dgain,
                           int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                           const whtmix_options *options)
{
    return module_backward_impl(x, w_in, whtmix::GAIN_FULL, gain, nullptr, nullptr, w_out, dy, dx,
                                dw_in, dw_out, dgain, nullptr, nullptr, B, N, C, dtype, stream,
                                options);
}

int whtmix_module_backward_separable(const void *x, const void *w_in, const float *log_gain_tokens,
                                     const float *log_gain_channels, const void *w_out,
                                     const void *dy, void *dx, float *dw_in, float *dw_out,
                                     float *d_log_gain_tokens, float *d_log_gain_channels,
                                     int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                                     const whtmix_options *options)
{
    return module_backward_impl(x, w_in, whtmix::GAIN_LOG_SEPARABLE, nullptr, log_gain_tokens,
                                log_gain_channels, w_out, dy, dx, dw_in, dw_out, nullptr,
                                d_log_gain_tokens, d_log_gain_channels, B, N, C, dtype, stream,
                                options);
}

int whtmix_backward(const void *x, const void *dy, const float *gain, void *dx, float *dgain,
                    int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                    const whtmix_options *options)
{
    return backward_impl(x, dy, whtmix::GAIN_FULL, gain, nullptr, nullptr, dx, dgain, nullptr,
                         nullptr, B, N, C, dtype, stream, options);
}

int whtmix_backward_separable(const void *x, const void *dy, const float *log_gain_tokens,
                              const float *log_gain_channels, void *dx,
                              float *d_log_gain_tokens, float *d_log_gain_channels, int64_t B,
                              int64_t N, int64_t C, int dtype, void *stream,
                              const whtmix_options *options)
{
    return backward_impl(x, dy, whtmix::GAIN_LOG_SEPARABLE, nullptr, log_gain_tokens,
                         log_gain_channels, dx, nullptr, d_log_gain_tokens, d_log_gain_channels,
                         B, N, C, dtype, stream, options);
}

int whtmix_module_forward(const void *x, const void *w_in, const float *gain, const void *w_out,
                          void *y, int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                          const whtmix_options *options)
{
    return module_impl(x, w_in, whtmix::GAIN_FULL, gain, nullptr, nullptr, w_out, y, B, N, C,
                       dtype, stream, options);
}

int whtmix_module_forward_separable(const void *x, const void *w_in, const float *log_gain_tokens,
                                    const float *log_gain_channels, const void *w_out, void *y,
                                    int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                                    const whtmix_options *options)
{
    return module_impl(x, w_in, whtmix::GAIN_LOG_SEPARABLE, nullptr, log_gain_tokens,
                       log_gain_channels, w_out, y, B, N, C, dtype, stream, options);
}

int whtmix_forward(const void *x, const float *gain, void *y, int64_t B, int64_t N, int64_t C,
                   int dtype, void *stream)
{
    return whtmix_forward_ex(x, gain, y, B, N, C, dtype, stream, nullptr);
}

int whtmix_forward_noalloc(const void *x, const float *gain, void *y, int64_t B, int64_t N,
                           int64_t C, int dtype, void *stream)
{
    return forward_impl(x, whtmix::GAIN_FULL, gain, nullptr, nullptr, y, B, N, C, dtype, stream,
                        nullptr, true);
}

const char *whtmix_status_string(int status)
{
    switch (status) {
    case WHTMIX_SUCCESS: return "success";
    case WHTMIX_ERROR_INVALID_VALUE: return "invalid value";
    case WHTMIX_ERROR_NOT_POWER_OF_TWO: return "C must be a power of two >= 1";
    case WHTMIX_ERROR_UNSUPPORTED_DTYPE: return "unsupported dtype";
    case WHTMIX_ERROR_MISALIGNED: return "x, y and gain must be 16-byte aligned";
    case WHTMIX_ERROR_OUT_OF_MEMORY: return "workspace allocation failed";
    case WHTMIX_ERROR_HIP: return "HIP runtime error";
    case WHTMIX_ERROR_TOO_LARGE:
        return "shape too large (N_pad*C <= 2^30, B*N_pad*C <= 2^37, module C <= 4096)";
    case WHTMIX_ERROR_DEVICE_TIMEOUT:
        return "a single-launch call gave up waiting for one of its passes";
    default: return "unknown status";
    }
}

const char *whtmix_last_error(void) { return g_last_error.c_str(); }

int whtmix_release_workspaces(void)
{
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    int st = WHTMIX_SUCCESS;
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) cur = -1;
    for (auto &kv : g_ws) {
        Workspace &w = kv.second;
        if (!w.ptr && !w.ctr) continue;
        if (hipSetDevice(kv.first.first) != hipSuccess ||
            hipStreamSynchronize(static_cast<hipStream_t>(kv.first.second)) != hipSuccess ||
            (w.ptr && hipFree(w.ptr) != hipSuccess) || (w.ctr && hipFree(w.ctr) != hipSuccess))
            st = WHTMIX_ERROR_HIP;
        w.ptr = nullptr;
        w.ctr = nullptr;
        w.bytes = 0;
    }
    g_ws.clear();
    if (cur >= 0) (void)hipSetDevice(cur);
    return st;
}

int whtmix_version(void) { return 10200; }

int whtmix_stream_status(void *stream)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    // Held while the error word is read and cleared, so that a concurrent
    // whtmix_release_workspaces cannot free the counter block meanwhile.
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    auto it = g_ws.find({dev, stream});
    uint32_t *ctr = it != g_ws.end() ? it->second.ctr : nullptr;
    if (!ctr) return WHTMIX_SUCCESS;
    // The sticky error word is the block's last word.
    uint32_t *sticky = ctr + whtmix::kCounterWords - 1;
    // Copies on the (idle) stream itself: the lock is not held across a
    // device-wide synchronisation.
    const hipStream_t st = static_cast<hipStream_t>(stream);
    uint32_t v = 0;
    e = hipMemcpyAsync(&v, sticky, sizeof(v), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "copy of the error word");
    if (v == 0) return WHTMIX_SUCCESS;
    const uint32_t zero = 0;
    e = hipMemcpyAsync(sticky, &zero, sizeof(zero), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "copy of the error word");
    return WHTMIX_ERROR_DEVICE_TIMEOUT;
}

}  // extern "C"
