/*
 * whtmix.h -- C ABI of the MI355X (gfx950) WHTMix token mixer.
 *
 * The mixer is the Walsh-Hadamard token mixer of "WHTMix: Efficient Stereo
 * Depth Estimation via Walsh-Hadamard Token Mixing", section III-B, eqs.
 * (2)-(3), in its joint per-frequency-gain form:
 *
 *     Y[b] = H_N (G o (H_N X[b] H_C)) H_C,      b = 0 .. B-1
 *
 *   X[b], Y[b]  N x C (tokens x channels), row-major, channels fastest;
 *   H_n         the orthonormal Sylvester-ordered Walsh-Hadamard matrix,
 *               entry (i, j) = (-1)^popcount(i & j) / sqrt(n), n = 2^k;
 *               H_n is symmetric and orthogonal, so H_n^{-1} = H_n;
 *   G           N_pad x C float32 per-frequency gain shared by every slice b
 *               ("o" is the element-wise product).
 *
 * C must be a power of two.  N may be any count >= 1: rows N .. N_pad-1 of
 * X, N_pad = 2^ceil(log2 N), are taken as zeros so that H_N acts on a
 * power-of-two length (section III-B), the mixer runs on the N_pad x C slice,
 * and Y keeps its first N rows.  For a power-of-two N, N_pad = N.
 *
 * The paper's own gains are log-domain vectors g_c (length C) and g_t
 * (length N_pad) applied by eq. (2) then eq. (3); that is this operation with
 * G[n][c] = exp(g_t[n]) * exp(g_c[c]), and whtmix_forward_separable() computes
 * it from the log gains directly.
 *
 * All computation runs in hand-written HIP kernels on the GPU.  Arithmetic is
 * float32 (bf16 inputs are widened exactly, bf16 outputs are rounded to
 * nearest even once at the end); the four orthonormal 1/sqrt factors are
 * applied together as the exact power of two 1/(N*C) at the gain multiply.
 *
 * Threading and streams: every entry point is safe to call from several host
 * threads.  Work is enqueued on the caller's stream and the call returns
 * without waiting for it.  The library keeps one float32 workspace of
 * B*N_pad*C*4 bytes per (device, stream) for shapes that need more than one
 * pass; it is allocated (or grown) on the first call that needs it, which
 * therefore synchronises that stream and is not safe inside HIP graph
 * capture.
 */
#ifndef WHTMIX_H
#define WHTMIX_H

#include <stdint.h>

#if defined(__GNUC__)
#define WHTMIX_API __attribute__((visibility("default")))
#else
#define WHTMIX_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of x and y (the gain is always float32). */
typedef enum whtmix_dtype {
    WHTMIX_DTYPE_F32 = 0,
    WHTMIX_DTYPE_BF16 = 1
} whtmix_dtype;

/* Return codes.  Every argument check runs on the host before any HIP call;
 * a rejected call enqueues nothing and writes nothing. */
typedef enum whtmix_status {
    WHTMIX_SUCCESS = 0,
    WHTMIX_ERROR_INVALID_VALUE = 1,    /* null pointer, B < 0, N < 1, partial
                                          x/y overlap, a gain overlapping y,
                                          bad option values */
    WHTMIX_ERROR_NOT_POWER_OF_TWO = 2, /* C not a power of two >= 1 */
    WHTMIX_ERROR_UNSUPPORTED_DTYPE = 3,
    WHTMIX_ERROR_MISALIGNED = 4,       /* x, y or gain not 16-byte aligned */
    WHTMIX_ERROR_OUT_OF_MEMORY = 5,    /* workspace allocation failed */
    WHTMIX_ERROR_HIP = 6,              /* HIP runtime / launch error; text in
                                          whtmix_last_error() */
    WHTMIX_ERROR_TOO_LARGE = 7,        /* N_pad*C > 2^30, sizes overflow, or
                                          module C > 4096 */
    WHTMIX_ERROR_DEVICE_TIMEOUT = 8    /* whtmix_stream_status only: a
                                          ONE_LAUNCH call on the stream gave
                                          up waiting for one of its passes
                                          (its output is not valid) */
} whtmix_status;

/* Execution plans.  AUTO picks by the padded slice size L = N_pad*C:
 *   L <= 2^10          one small workgroup per slice, all stages in LDS;
 *   2^11 <= L <= 2^15  FUSED: one workgroup per slice, a single pass; for
 *                      L = 2^15 up to 48 slices TWO_PASS instead;
 *   L = 2^16           WAVE_TILES up to 3 slices, TWO_PASS from 4 to 16,
 *                      FUSED (two register sets) from 48 slices, THREE_PASS
 *                      between;
 *   L >= 2^17          THREE_PASS: forward over the low bits of the flat
 *                      index, then forward over the high bits + gain +
 *                      inverse over the high bits, then inverse over the low
 *                      bits, exchanging through the workspace.
 * WAVE_TILES runs the same three passes on one-wave tiles of 2^9 elements
 * whose butterflies stay inside the wave (DPP and lane-swap exchanges, no
 * LDS): three launches of 2^(K-9) workgroups per slice; 2^12 <= L <= 2^16
 * and N*C a multiple of 8 (AUTO falls back to the plans above otherwise);
 * forced, B*L < 2^35 besides (WHTMIX_ERROR_TOO_LARGE beyond).
 * TWO_PASS (L = 2^15 or 2^16, N*C a multiple of 8) replaces WAVE_TILES's
 * first two launches by one: each of a slice's 2^(K-12) workgroups reads the
 * whole slice and forms its share of the low-bit transform as a signed sum
 * of the slice's blocks, then runs the high bits, the gain and their
 * inverse; WAVE_TILES's last launch follows.  B rounded up to a multiple of
 * 8, times L, must stay below 2^35.
 * ONE_LAUNCH (never chosen by AUTO) runs WAVE_TILES's three passes in a
 * single cooperative launch, ordered by per-slice counters in a small
 * per-stream block; B <= 2046 besides.  On MI355X it is slower than the plans
 * AUTO picks: a cooperative launch alone costs about 20 us, and a hand-off
 * between workgroups through memory costs more than a kernel boundary.
 * THREE_PASS may also be forced for 2^12 <= L <= 2^16 (tests compare it with
 * FUSED on the same shapes).  The backward pass and the block take FUSED
 * for slices up to 2^15 and THREE_PASS from 2^16 whatever the forward plan. */
typedef enum whtmix_plan {
    WHTMIX_PLAN_AUTO = 0,
    WHTMIX_PLAN_SMALL = 1,
    WHTMIX_PLAN_FUSED = 2,
    WHTMIX_PLAN_THREE_PASS = 3,
    WHTMIX_PLAN_ONE_LAUNCH = 4,
    WHTMIX_PLAN_WAVE_TILES = 5,
    WHTMIX_PLAN_TWO_PASS = 6
} whtmix_plan;

typedef struct whtmix_options {
    int plan;          /* whtmix_plan; WHTMIX_PLAN_AUTO = 0 */
    /* Optional hipEvent_t handles (NULL to skip).  events[0] is recorded on
     * the stream before the first kernel and events[i] after the i-th kernel
     * of the plan (at most 3 kernels).  Used for per-kernel timing. */
    void *events[4];
    /* ONE_LAUNCH: polls of the kernel's counter waits before the call gives
     * up (0 = the default, about a second or two).  A call that gives up
     * exits normally with an invalid output and raises the stream's error
     * word (whtmix_stream_status).  Tests force that path with a tiny
     * limit. */
    uint32_t spin_limit;
} whtmix_options;

/* Describes how a shape would run (no GPU work, no allocation).  plan,
 * kernels and workspace_bytes are whtmix_forward's; the backward pass and the
 * block run 2^16-element slices, whose forward is FUSED, with the three-pass
 * plan (and its workspace). */
typedef struct whtmix_plan_info {
    int plan;             /* resolved whtmix_plan (never AUTO) */
    int kernels;          /* kernels launched per call (1 or 3) */
    int log2_slice;       /* K = log2(N*C) */
    int outer_bits;       /* THREE_PASS, WAVE_TILES, ONE_LAUNCH: flat-index bits of the
                             outer passes */
    int run_bits;         /* THREE_PASS, WAVE_TILES, ONE_LAUNCH: log2 of the contiguous run carried
                             by the middle pass */
    int64_t workspace_bytes; /* float32 workspace this call needs */
    int64_t padded_tokens;   /* N_pad */
    /* How whtmix_module_forward runs this shape: 0 SMALL (projections on the
     * vector ALUs), 1 projections fused into the mixer's kernels on the
     * matrix cores, 2 projection kernels around the float32 mixer; -1 when C
     * exceeds the block's limit. */
    int module_path;
    int module_outer_bits;   /* THREE_PASS: the block's outer-pass bits */
    /* 1 when whtmix_module_backward runs its projections inside the mixer
     * backward's passes (given B > 0 and a requested gain gradient); its
     * events then bracket [transforms of Z and dZ', gain gradient], [Z',
     * dW_out], [dX, dW_in] instead of [Z, Z', dZ', dW_out], [the mixer's
     * gradients], [dX, dW_in]. */
    int module_backward_fused;
} whtmix_plan_info;

/*
 * whtmix_forward -- y[b] = H_N (G o (H_N x[b] H_C)) H_C for b in [0, B)
 * (section III-B, eqs. (2)-(3), joint gain).
 *
 *   x      device pointer, [B][N][C] contiguous elements of `dtype`
 *          (read only).  May equal y exactly (in place); any other overlap
 *          with y is rejected.
 *   gain   device pointer, [N_pad][C] contiguous float32 (linear gains),
 *          shared by all b; must not overlap y.
 *   y      device pointer, [B][N][C] contiguous elements of `dtype` (written).
 *   B      number of independent slices; B == 0 is a no-op (pointers are not
 *          inspected).
 *   N, C   tokens (>= 1) and channels (a power of two >= 1), N_pad*C <= 2^30.
 *   dtype  whtmix_dtype of x and y.
 *   stream hipStream_t to enqueue on (NULL = the null stream).
 *
 * The caller owns x, gain and y and keeps them alive until the stream work
 * is done.  Pointers must be 16-byte aligned.  Returns a whtmix_status.
 * Kernel faults surface asynchronously through the stream like any HIP op.
 */
WHTMIX_API int whtmix_forward(const void *x, const float *gain, void *y,
                   int64_t B, int64_t N, int64_t C, int dtype, void *stream);

/*
 * whtmix_forward_noalloc -- whtmix_forward for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, result, plan (AUTO) and checks as
 * whtmix_forward, but the workspace of the three-pass, two-pass and wave-tile
 * plans is a fixed 32 MiB device array inside the library (one per device, held until the process ends) instead
 * of the per-stream workspace, and the call allocates nothing: no hipMalloc,
 * no hipFree, no stream synchronisation.  Limit: shapes whose plan needs a
 * workspace must have B * N_pad * C <= 2^23; larger ones return
 * WHTMIX_ERROR_TOO_LARGE (text in whtmix_last_error()) with nothing
 * enqueued.  Every call on a device shares that device's array, so calls
 * that overlap on one device (on different streams or host threads) race;
 * serialise them.
 */
WHTMIX_API int whtmix_forward_noalloc(const void *x, const float *gain, void *y,
                           int64_t B, int64_t N, int64_t C, int dtype, void *stream);

/* As whtmix_forward, with options (NULL = defaults). */
WHTMIX_API int whtmix_forward_ex(const void *x, const float *gain, void *y,
                      int64_t B, int64_t N, int64_t C, int dtype, void *stream,
                      const whtmix_options *options);

/*
 * whtmix_forward_separable -- the paper's parametrisation, eq. (2) then
 * eq. (3):  Z <- H_C^{-1}(exp(g_c) o H_C Z) along channels, then
 *           Z <- H_N^{-1}(exp(g_t) o H_N Z) along tokens,
 * i.e. whtmix_forward with G[n][c] = exp(g_t[n]) * exp(g_c[c]).  The gain of
 * each frequency is formed on the device as exp(g_t[n] + g_c[c]), so the
 * only gain traffic is the two small vectors.
 *
 *   log_gain_tokens    device pointer, [N_pad] float32 log gains g_t
 *   log_gain_channels  device pointer, [C] float32 log gains g_c
 * Both are 16-byte aligned and must not overlap y (zero log gains, the
 * paper's initialisation, give Y = X).  Other arguments, options and return
 * codes as whtmix_forward_ex (options may be NULL).
 */
WHTMIX_API int whtmix_forward_separable(const void *x, const float *log_gain_tokens,
                             const float *log_gain_channels, void *y,
                             int64_t B, int64_t N, int64_t C, int dtype,
                             void *stream, const whtmix_options *options);

/*
 * whtmix_backward -- gradients through whtmix_forward for an upstream
 * gradient dy = dL/dy (the paper trains the gains, section IV-A).  With the
 * orthonormal transforms T(v) = H_Npad vpad H_C of zero-padded slices:
 *     dx[b] = H_N (G o T(dy[b])) H_C, first N rows (the mixer is
 *             self-adjoint, so this is whtmix_forward applied to dy);
 *     dgain = sum over b of T(x[b]) o T(dy[b])        ([N_pad][C] float32).
 *
 *   x, dy  device pointers, [B][N][C] elements of `dtype` (x is not read when
 *          dgain is NULL).
 *   gain   [N_pad][C] float32, as passed to the forward call.
 *   dx     [B][N][C] of `dtype`, or NULL to skip; may be dy itself.
 *   dgain  [N_pad][C] float32, overwritten (not accumulated), or NULL to skip.
 * At least one of dx, dgain must be non-NULL.  No output may overlap an
 * input or another output (except dx == dy).  With B == 0 dgain is filled
 * with zeros.  The gain gradient is summed over the batch in a fixed order,
 * so results are bitwise reproducible.  The call uses a float32 workspace of
 * up to 2*B*N_pad*C (+ partial sums) floats; other conventions and options as
 * whtmix_forward_ex (events: [0] before, [1] after the gain gradient, [2]
 * after dx).  With the three-pass plan and both outputs requested, the two
 * gradients share dy's transform: the gain gradient is complete at [1] and
 * only dx's last pass runs between [1] and [2].
 */
WHTMIX_API int whtmix_backward(const void *x, const void *dy, const float *gain,
                    void *dx, float *dgain, int64_t B, int64_t N, int64_t C,
                    int dtype, void *stream, const whtmix_options *options);

/*
 * whtmix_backward_separable -- gradients through whtmix_forward_separable:
 *     dx                as whtmix_backward with G[n][c] = exp(g_t[n] + g_c[c]),
 *     d_log_gain_tokens[n]   = sum over c of dG[n][c] G[n][c]   ([N_pad]),
 *     d_log_gain_channels[c] = sum over n of dG[n][c] G[n][c]   ([C]),
 * (the chain rule through exp).  The two log-gain gradients are both NULL or
 * both non-NULL; everything else as whtmix_backward.
 */
WHTMIX_API int whtmix_backward_separable(const void *x, const void *dy,
                              const float *log_gain_tokens,
                              const float *log_gain_channels, void *dx,
                              float *d_log_gain_tokens,
                              float *d_log_gain_channels, int64_t B,
                              int64_t N, int64_t C, int dtype, void *stream,
                              const whtmix_options *options);

/*
 * whtmix_module_forward -- the whole block of section III-B, eqs. (1)-(4),
 * with the joint gain:
 *     Z = X[b] W_in;   Z <- H_N (G o (H_N Z H_C)) H_C;   Y[b] = Z W_out
 * (Z zero-padded to N_pad rows before H_N, Y cropped to the first N rows),
 * the drop-in replacement of the self-attention block with its projections.
 *
 *   x      [B][N][C] elements of `dtype`; may equal y exactly (in place).
 *   w_in   [C][C] elements of `dtype`, row-major: Z[n][j] = sum_i X[n][i]
 *          W_in[i][j].
 *   gain   [N_pad][C] float32 linear gains (as whtmix_forward).
 *   w_out  [C][C] elements of `dtype`: Y[n][j] = sum_i Z[n][i] W_out[i][j].
 *   y      [B][N][C] elements of `dtype` (written).
 * C is a power of two <= 4096 (WHTMIX_ERROR_TOO_LARGE above).  Inputs must
 * not overlap y except x == y.  Arithmetic is float32: for bf16 the products
 * X W_in are exact, Z' W_out uses a two-term bf16 split of Z' (relative
 * residual below 2^-17), and y is rounded to nearest even once.  For
 * 16 <= C <= 128, and for bf16 C = 256 from N_pad*C = 2^17, the projections
 * run on the matrix cores inside the mixer's first and last kernels (three
 * kernels plus a small weight-repacking kernel for N_pad*C > 2^15;
 * whtmix_plan_describe's module_path says which); other shapes run separate
 * projection kernels around the float32 mixer.  Workspace: the mixer's, plus
 * 2*C*C elements of packed weights or B*N*C floats of Z.  Other conventions, plans and options as
 * whtmix_forward_ex (events: for the three-pass plan around each of its
 * three passes, otherwise [0] before and [1] after the call's kernels).
 */
WHTMIX_API int whtmix_module_forward(const void *x, const void *w_in,
                          const float *gain, const void *w_out, void *y,
                          int64_t B, int64_t N, int64_t C, int dtype,
                          void *stream, const whtmix_options *options);

/*
 * whtmix_module_forward_separable -- whtmix_module_forward with the paper's
 * log-domain gains (eqs. (2)-(3)): log_gain_tokens [N_pad] and
 * log_gain_channels [C] float32, as whtmix_forward_separable.
 */
WHTMIX_API int whtmix_module_forward_separable(const void *x, const void *w_in,
                                    const float *log_gain_tokens,
                                    const float *log_gain_channels,
                                    const void *w_out, void *y, int64_t B,
                                    int64_t N, int64_t C, int dtype,
                                    void *stream,
                                    const whtmix_options *options);

/*
 * whtmix_module_backward -- gradients through whtmix_module_forward for an
 * upstream gradient dy = dL/dY (the paper trains the block, section IV-A):
 *     dZ' = dY W_out^T,            dW_out = sum over b of Z'^T dY,
 *     dZ, dgain = the mixer's gradients (whtmix_backward) at (Z, dZ'),
 *     dX = dZ W_in^T,              dW_in  = sum over b of X^T dZ,
 * with Z = X W_in and Z' = mixer(Z) recomputed in float32.  For 16 <= C <=
 * 128 on three-pass slices up to 2^25 elements, and bf16 C = 256 on
 * 2^26..2^28 (with a requested gain gradient), the projections run inside
 * the mixer backward's passes and Z and dZ' are never stored
 * (whtmix_plan_describe's module_backward_fused).
 *
 *   x, dy         [B][N][C] elements of `dtype`.
 *   w_in, w_out   [C][C] elements of `dtype`, as passed to the forward call.
 *   gain          [N_pad][C] float32.
 *   dx            [B][N][C] of `dtype` (written); may be dy itself.
 *   dw_in, dw_out [C][C] float32, overwritten.
 *   dgain         [N_pad][C] float32, overwritten, or NULL to skip.
 * No output may overlap an input or another output (except dx == dy); B*N <
 * 2^31.  Weight gradients are summed over row chunks in a fixed order, so
 * results are bitwise reproducible.  Workspace: 3*B*N*C floats plus the
 * mixer's forward and backward workspaces, 3*C*C packed weight elements and
 * the weight-gradient partial sums.  Other conventions as
 * whtmix_module_forward (events: [0] before, then after each phase: [1]
 * dW_out, [2] the mixer's gradients, [3] dX and dW_in; with the projections
 * inside the mixer's passes [1] the gain gradient, [2] dW_out, [3] dX and
 * dW_in).
 */
WHTMIX_API int whtmix_module_backward(const void *x, const void *w_in,
                           const float *gain, const void *w_out,
                           const void *dy, void *dx, float *dw_in,
                           float *dw_out, float *dgain, int64_t B, int64_t N,
                           int64_t C, int dtype, void *stream,
                           const whtmix_options *options);

/*
 * whtmix_module_backward_separable -- as whtmix_module_backward for the
 * block with log-domain gains: d_log_gain_tokens [N_pad] and
 * d_log_gain_channels [C] float32 (both NULL or both non-NULL), as
 * whtmix_backward_separable.
 */
WHTMIX_API int whtmix_module_backward_separable(const void *x, const void *w_in,
                                     const float *log_gain_tokens,
                                     const float *log_gain_channels,
                                     const void *w_out, const void *dy,
                                     void *dx, float *dw_in, float *dw_out,
                                     float *d_log_gain_tokens,
                                     float *d_log_gain_channels, int64_t B,
                                     int64_t N, int64_t C, int dtype,
                                     void *stream,
                                     const whtmix_options *options);

/* Fills *info with the plan whtmix_forward_ex would use.  Validates the
 * shape, dtype and options exactly as the forward call does (pointers are
 * not needed).  Returns a whtmix_status. */
WHTMIX_API int whtmix_plan_describe(int64_t B, int64_t N, int64_t C, int dtype,
                         const whtmix_options *options,
                         whtmix_plan_info *info);

/* Static description of a status code (never NULL). */
WHTMIX_API const char *whtmix_status_string(int status);

/* Text of the last WHTMIX_ERROR_HIP / OUT_OF_MEMORY on the calling thread
 * ("" if none). */
WHTMIX_API const char *whtmix_last_error(void);

/* Synchronises every stream that owns a workspace and frees all workspaces.
 * Returns a whtmix_status. */
WHTMIX_API int whtmix_release_workspaces(void);

/* Synchronises `stream` (hipStream_t) on the current device, then reports
 * and clears the error word its ONE_LAUNCH calls raise: WHTMIX_SUCCESS when
 * every ONE_LAUNCH call since the last check completed, or
 * WHTMIX_ERROR_DEVICE_TIMEOUT when one gave up waiting for a pass (its
 * output is invalid; later calls are unaffected).  Other plans never raise
 * it.  Returns WHTMIX_ERROR_HIP if the synchronisation fails. */
WHTMIX_API int whtmix_stream_status(void *stream);

/* Library version as major*10000 + minor*100 + patch. */
WHTMIX_API int whtmix_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WHTMIX_H */
