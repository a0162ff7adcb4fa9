/*
 * WHTMix CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, double-precision statement of the Walsh-Hadamard token mixer
 * (Method, section III-B, eqs. (2)-(3)).  Only the test suite, the smoke check
 * and the CPU-baseline leg of the benchmark may load this library; the product
 * path (the HIP library) never calls it, and the two share no code, headers or
 * build steps.
 *
 * What the paper fixes:
 *   - H is the orthonormal Walsh-Hadamard transform: the Sylvester-Hadamard
 *     matrix divided by sqrt(n), n a power of two, applied by an O(n log n)
 *     butterfly (section III-B, first paragraph).
 *   - Sylvester order is natural Hadamard order: H_1 = [1],
 *     H_2n = [[H_n, H_n], [H_n, -H_n]], so entry (i, j) is
 *     (-1)^popcount(i & j) / sqrt(n).  No bit reversal is involved.
 *   - Channel mixing (eq. 2) acts along each token row of X in R^{N x C};
 *     token mixing (eq. 3) acts along each channel column.
 *   - Both transforms are orthonormal and H^{-1} = H (H is symmetric and
 *     orthogonal), so the "inverse" transform is the same butterfly.
 *
 * The mixer computed here (joint-gain form):
 *     Y[b] = H_N (G o (H_N X[b] H_C)) H_C,   b = 0 .. B-1,
 * with G[N, C] a per-frequency gain shared by all batch slices and "o" the
 * element-wise product.  The paper's own parametrisation, log-domain gains
 * g_c (length C) and g_t (length N) applied by eq. (2) then eq. (3), is
 * oracle_whtmix_separable(); it equals the joint form with
 * G[n][c] = exp(g_t[n]) * exp(g_c[c]) (rank one).
 *
 * Token padding: C must be a power of two; N may be any count >= 1.  As in
 * section III-B, the token axis is zero-padded to P = 2^ceil(log2 N) rows
 * before the transforms; the mixer runs on the P x C slice and the first N
 * rows are kept.  The gains then cover P token frequencies.
 *
 * Layout: x, y are [B][N][C] row-major (C fastest), g is [P][C] row-major.
 * Every per-vector operation runs in a fixed order, so the output is bitwise
 * independent of the OpenMP thread count.
 */
#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

/* Unnormalised Sylvester butterfly, in place, on the n values v[0], v[s],
 * v[2s], ...: after the loop v holds H_n v with H_n the +/-1 Sylvester matrix
 * (section III-B).  Each stage pairs index j with j + h inside blocks of 2h
 * and replaces (a, b) by (a + b, a - b). */
static void fwht_strided(double *v, long n, long s)
{
    for (long h = 1; h < n; h *= 2) {
        for (long i = 0; i < n; i += 2 * h) {
            for (long j = i; j < i + h; ++j) {
                double a = v[j * s];
                double b = v[(j + h) * s];
                v[j * s] = a + b;
                v[(j + h) * s] = a - b;
            }
        }
    }
}

/* Orthonormal transform: the butterfly followed by the 1/sqrt(n) factor that
 * makes H orthonormal (section III-B). */
static void wht_orthonormal(double *v, long n, long s)
{
    fwht_strided(v, n, s);
    double f = 1.0 / sqrt((double)n);
    for (long j = 0; j < n; ++j)
        v[j * s] *= f;
}

/* Z <- Z H_C: transform every token row along the channel axis. */
static void channel_transform(double *z, long N, long C)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; ++n)
        wht_orthonormal(z + n * C, C, 1);
}

/* Z <- H_N Z: transform every channel column along the token axis. */
static void token_transform(double *z, long N, long C)
{
#pragma omp parallel for schedule(static)
    for (long c = 0; c < C; ++c)
        wht_orthonormal(z + c, N, C);
}

static int is_pow2(long n) { return n >= 1 && (n & (n - 1)) == 0; }

/* Smallest power of two >= n: the padded token count. */
static long padded(long n)
{
    long p = 1;
    while (p < n)
        p *= 2;
    return p;
}

/* z <- x[b] followed by P - N zero rows (the zero-padded token axis). */
static void load_padded(double *z, const double *xb, long N, long P, long C)
{
    memcpy(z, xb, (size_t)(N * C) * sizeof(double));
    memset(z + N * C, 0, (size_t)((P - N) * C) * sizeof(double));
}

/* Joint-gain mixer, Y[b] = first N rows of H_P (G o (H_P Xpad[b] H_C)) H_C.
 * g is [P][C].  Returns 0 on success, -1 on a bad argument (null pointer,
 * B < 0, N < 1, C not a power of two, allocation failure). */
int oracle_whtmix(const double *x, const double *g, double *y,
                  long B, long N, long C)
{
    if (!x || !g || !y || B < 0 || N < 1 || !is_pow2(C))
        return -1;
    const long P = padded(N);
    double *z = malloc((size_t)(P * C) * sizeof(double));
    if (!z)
        return -1;
    for (long b = 0; b < B; ++b) {
        load_padded(z, x + b * N * C, N, P, C);
        /* forward: T = H_P Z H_C */
        channel_transform(z, P, C);
        token_transform(z, P, C);
        /* per-frequency gain */
        for (long i = 0; i < P * C; ++i)
            z[i] *= g[i];
        /* inverse (H^{-1} = H): Y = H_P T H_C */
        token_transform(z, P, C);
        channel_transform(z, P, C);
        memcpy(y + b * N * C, z, (size_t)(N * C) * sizeof(double));
    }
    free(z);
    return 0;
}

/* The paper's literal parametrisation, eq. (2) then eq. (3):
 *   Z <- H_C^{-1}( exp(g_c) o H_C(Z) )   along channels, per token row,
 *   Z <- H_P^{-1}( exp(g_t) o H_P(Z) )   along tokens, per channel column,
 * with g_c (length C) and g_t (length P) log-domain gains.  Same return
 * convention as oracle_whtmix(). */
int oracle_whtmix_separable(const double *x, const double *g_t,
                            const double *g_c, double *y,
                            long B, long N, long C)
{
    if (!x || !g_t || !g_c || !y || B < 0 || N < 1 || !is_pow2(C))
        return -1;
    const long P = padded(N);
    double *z = malloc((size_t)(P * C) * sizeof(double));
    if (!z)
        return -1;
    for (long b = 0; b < B; ++b) {
        load_padded(z, x + b * N * C, N, P, C);
        /* eq. (2): channel mixing */
        channel_transform(z, P, C);
        for (long n = 0; n < P; ++n)
            for (long c = 0; c < C; ++c)
                z[n * C + c] *= exp(g_c[c]);
        channel_transform(z, P, C);
        /* eq. (3): token mixing */
        token_transform(z, P, C);
        for (long n = 0; n < P; ++n)
            for (long c = 0; c < C; ++c)
                z[n * C + c] *= exp(g_t[n]);
        token_transform(z, P, C);
        memcpy(y + b * N * C, z, (size_t)(N * C) * sizeof(double));
    }
    free(z);
    return 0;
}

/* Z = X W for one slice: Z[n][j] = sum over i of X[n][i] W[i][j] (W is
 * [C][C] row-major), the projections of eqs. (1) and (4).  Each Z[n][j] is
 * summed over i in ascending order; the loops run i outside j only so that W
 * is read along its rows. */
static void project(const double *x, const double *w, double *z, long N, long C)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; ++n) {
        double *zn = z + n * C;
        for (long j = 0; j < C; ++j)
            zn[j] = 0.0;
        for (long i = 0; i < C; ++i) {
            const double xi = x[n * C + i];
            for (long j = 0; j < C; ++j)
                zn[j] += xi * w[i * C + j];
        }
    }
}

/* The full WHTMix block, eqs. (1)-(4): Z = X W_in; the token mixer on Z
 * (joint gain g [P][C], or separable log gains when g is NULL and g_t, g_c
 * are given); Y = Z W_out.  Same return convention as oracle_whtmix(). */
static int module_impl(const double *x, const double *w_in, const double *g,
                       const double *g_t, const double *g_c,
                       const double *w_out, double *y, long B, long N, long C)
{
    if (!x || !w_in || !w_out || !y || B < 0 || N < 1 || !is_pow2(C))
        return -1;
    double *z = malloc((size_t)(N * C) * sizeof(double));
    double *m = malloc((size_t)(N * C) * sizeof(double));
    if (!z || !m) {
        free(z);
        free(m);
        return -1;
    }
    int rc = 0;
    for (long b = 0; b < B && rc == 0; ++b) {
        project(x + b * N * C, w_in, z, N, C);                     /* eq. (1) */
        rc = g ? oracle_whtmix(z, g, m, 1, N, C)                   /* eqs. (2)-(3) */
               : oracle_whtmix_separable(z, g_t, g_c, m, 1, N, C);
        if (rc == 0)
            project(m, w_out, y + b * N * C, N, C);                /* eq. (4) */
    }
    free(z);
    free(m);
    return rc;
}

int oracle_whtmix_module(const double *x, const double *w_in, const double *g,
                         const double *w_out, double *y, long B, long N, long C)
{
    if (!g)
        return -1;
    return module_impl(x, w_in, g, NULL, NULL, w_out, y, B, N, C);
}

int oracle_whtmix_module_separable(const double *x, const double *w_in,
                                   const double *g_t, const double *g_c,
                                   const double *w_out, double *y,
                                   long B, long N, long C)
{
    if (!g_t || !g_c)
        return -1;
    return module_impl(x, w_in, NULL, g_t, g_c, w_out, y, B, N, C);
}

/* Gradients through the joint-gain mixer (the paper trains the gains,
 * section IV-A).  For a loss with upstream gradient dY = dL/dY, and
 *     T_x[b]  = H_P Xpad[b] H_C,   T_dy[b] = H_P dYpad[b] H_C
 * (orthonormal transforms of the zero-padded slices):
 *     dX[b] = first N rows of H_P (G o T_dy[b]) H_C
 *             (the mixer is self-adjoint: H symmetric, G diagonal),
 *     dG    = sum over b of T_x[b] o T_dy[b].
 * dx or dg may be NULL to skip that output.  Same return convention as
 * oracle_whtmix(). */
int oracle_whtmix_grad(const double *x, const double *dy, const double *g,
                       double *dx, double *dg, long B, long N, long C)
{
    if (!x || !dy || !g || B < 0 || N < 1 || !is_pow2(C))
        return -1;
    if (dx && oracle_whtmix(dy, g, dx, B, N, C) != 0)
        return -1;
    if (!dg)
        return 0;
    const long P = padded(N);
    double *tx = malloc((size_t)(P * C) * sizeof(double));
    double *td = malloc((size_t)(P * C) * sizeof(double));
    if (!tx || !td) {
        free(tx);
        free(td);
        return -1;
    }
    memset(dg, 0, (size_t)(P * C) * sizeof(double));
    for (long b = 0; b < B; ++b) {
        load_padded(tx, x + b * N * C, N, P, C);
        channel_transform(tx, P, C);
        token_transform(tx, P, C);
        load_padded(td, dy + b * N * C, N, P, C);
        channel_transform(td, P, C);
        token_transform(td, P, C);
        for (long i = 0; i < P * C; ++i)
            dg[i] += tx[i] * td[i];
    }
    free(tx);
    free(td);
    return 0;
}

/* Gradients through the separable form (eqs. (2)-(3)), whose joint gain is
 * G[n][c] = exp(g_t[n]) exp(g_c[c]):
 *     dX         as oracle_whtmix_grad with that G,
 *     dg_t[n]  = sum over c of dG[n][c] G[n][c],
 *     dg_c[c]  = sum over n of dG[n][c] G[n][c]   (chain rule through exp).
 * Any of dx, dg_t, dg_c may be NULL (dg_t and dg_c together). */
int oracle_whtmix_grad_separable(const double *x, const double *dy,
                                 const double *g_t, const double *g_c,
                                 double *dx, double *dg_t, double *dg_c,
                                 long B, long N, long C)
{
    if (!x || !dy || !g_t || !g_c || B < 0 || N < 1 || !is_pow2(C))
        return -1;
    if (dx && oracle_whtmix_separable(dy, g_t, g_c, dx, B, N, C) != 0)
        return -1;
    if (!dg_t || !dg_c)
        return 0;
    const long P = padded(N);
    double *G = malloc((size_t)(P * C) * sizeof(double));
    double *dG = malloc((size_t)(P * C) * sizeof(double));
    if (!G || !dG) {
        free(G);
        free(dG);
        return -1;
    }
    for (long n = 0; n < P; ++n)
        for (long c = 0; c < C; ++c)
            G[n * C + c] = exp(g_t[n]) * exp(g_c[c]);
    if (oracle_whtmix_grad(x, dy, G, NULL, dG, B, N, C) != 0) {
        free(G);
        free(dG);
        return -1;
    }
    for (long n = 0; n < P; ++n) {
        double s = 0.0;
        for (long c = 0; c < C; ++c)
            s += dG[n * C + c] * G[n * C + c];
        dg_t[n] = s;
    }
    for (long c = 0; c < C; ++c) {
        double s = 0.0;
        for (long n = 0; n < P; ++n)
            s += dG[n * C + c] * G[n * C + c];
        dg_c[c] = s;
    }
    free(G);
    free(dG);
    return 0;
}

/* Backward through a projection: Z[n][i] = sum over j of X[n][j] W[i][j],
 * i.e. Z = X W^T with W [C][C] row-major (each sum over j ascending). */
static void project_t(const double *x, const double *w, double *z, long N, long C)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; ++n)
        for (long i = 0; i < C; ++i) {
            double s = 0.0;
            for (long j = 0; j < C; ++j)
                s += x[n * C + j] * w[i * C + j];
            z[n * C + i] = s;
        }
}

/* Weight gradient of a projection: acc[i][j] += sum over n of a[n][i] b[n][j]
 * (acc = A^T B; each row i of acc belongs to one thread, n ascending). */
static void accumulate_at_b(const double *a, const double *b, double *acc, long N, long C)
{
#pragma omp parallel for schedule(static)
    for (long i = 0; i < C; ++i)
        for (long n = 0; n < N; ++n) {
            const double ai = a[n * C + i];
            for (long j = 0; j < C; ++j)
                acc[i * C + j] += ai * b[n * C + j];
        }
}

/* Gradients of the whole block, eqs. (1)-(4), for an upstream gradient dY:
 *   Z = X W_in, Z' = mixer(Z), Y = Z' W_out  (forward, recomputed here);
 *   dZ' = dY W_out^T;      dW_out = sum over b of Z'^T dY;
 *   dZ and the gain gradient from the mixer's own gradient at (Z, dZ');
 *   dX = dZ W_in^T;        dW_in = sum over b of X^T dZ.
 * Joint gain g [P][C] (dg), or separable log gains when g is NULL (dgt, dgc). */
static int module_grad_impl(const double *x, const double *w_in, const double *g,
                            const double *g_t, const double *g_c, const double *w_out,
                            const double *dy, double *dx, double *dw_in, double *dw_out,
                            double *dg, double *dgt, double *dgc, long B, long N, long C)
{
    if (!x || !w_in || !w_out || !dy || !dx || !dw_in || !dw_out || B < 0 || N < 1 ||
        !is_pow2(C))
        return -1;
    const size_t n = (size_t)(B * N * C);
    double *z = malloc((n ? n : 1) * sizeof(double));
    double *zp = malloc((n ? n : 1) * sizeof(double));
    double *dzp = malloc((n ? n : 1) * sizeof(double));
    double *dz = malloc((n ? n : 1) * sizeof(double));
    int rc = (z && zp && dzp && dz) ? 0 : -1;
    const long S = N * C;
    for (long b = 0; b < B && rc == 0; ++b)
        project(x + b * S, w_in, z + b * S, N, C);                          /* eq. (1) */
    if (rc == 0)
        rc = g ? oracle_whtmix(z, g, zp, B, N, C)                          /* eqs. (2)-(3) */
               : oracle_whtmix_separable(z, g_t, g_c, zp, B, N, C);
    for (long b = 0; b < B && rc == 0; ++b)
        project_t(dy + b * S, w_out, dzp + b * S, N, C);                   /* through eq. (4) */
    if (rc == 0) {
        for (long i = 0; i < C * C; ++i)
            dw_out[i] = 0.0;
        for (long b = 0; b < B; ++b)
            accumulate_at_b(zp + b * S, dy + b * S, dw_out, N, C);
        rc = g ? oracle_whtmix_grad(z, dzp, g, dz, dg, B, N, C)
               : oracle_whtmix_grad_separable(z, dzp, g_t, g_c, dz, dgt, dgc, B, N, C);
    }
    for (long b = 0; b < B && rc == 0; ++b)
        project_t(dz + b * S, w_in, dx + b * S, N, C);                     /* through eq. (1) */
    if (rc == 0) {
        for (long i = 0; i < C * C; ++i)
            dw_in[i] = 0.0;
        for (long b = 0; b < B; ++b)
            accumulate_at_b(x + b * S, dz + b * S, dw_in, N, C);
    }
    free(z);
    free(zp);
    free(dzp);
    free(dz);
    return rc;
}

int oracle_whtmix_module_grad(const double *x, const double *w_in, const double *g,
                              const double *w_out, const double *dy, double *dx,
                              double *dw_in, double *dw_out, double *dg, long B, long N,
                              long C)
{
    if (!g || !dg)
        return -1;
    return module_grad_impl(x, w_in, g, NULL, NULL, w_out, dy, dx, dw_in, dw_out, dg, NULL,
                            NULL, B, N, C);
}

int oracle_whtmix_module_grad_separable(const double *x, const double *w_in,
                                        const double *g_t, const double *g_c,
                                        const double *w_out, const double *dy, double *dx,
                                        double *dw_in, double *dw_out, double *dgt,
                                        double *dgc, long B, long N, long C)
{
    if (!g_t || !g_c || !dgt || !dgc)
        return -1;
    return module_grad_impl(x, w_in, NULL, g_t, g_c, w_out, dy, dx, dw_in, dw_out, NULL, dgt,
                            dgc, B, N, C);
}

/* Bare unnormalised butterfly over a contiguous vector, exported so that the
 * tests can pin the transform itself against a dense Sylvester matrix. */
int oracle_fwht(double *v, long n)
{
    if (!v || !is_pow2(n))
        return -1;
    fwht_strided(v, n, 1);
    return 0;
}

/* Number of OpenMP threads a parallel region of the oracle uses. */
int oracle_threads(void)
{
    return omp_get_max_threads();
}

/* Sets the number of OpenMP threads later calls use (n >= 1); returns the
 * previous count.  Per-vector operation order does not depend on it, so the
 * results are bitwise the same at any count. */
int oracle_set_threads(int n)
{
    const int prev = omp_get_max_threads();
    if (n >= 1)
        omp_set_num_threads(n);
    return prev;
}
