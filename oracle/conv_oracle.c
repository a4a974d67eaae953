/*
 * conv_oracle.c -- fp64 CPU reference for 2-D convolution in its three
 * training passes.  TEST INFRASTRUCTURE ONLY: this file is compiled and
 * called by the test-suite, by the smoke check and by the CPU-baseline leg
 * of the benchmark.  The GPU library never links, includes or calls it,
 * and it shares no header, table or helper with the GPU library.
 *
 * What it computes.  The paper states convolution only as an API call
 * (Sec. 3.2, Listings 4-5: convolution(x, base_axis=1, outmaps, kernel)),
 * with the batch on axis 0 and channels on axis 1, and trains it with
 * back-propagation (Sec. 2.1) in mixed precision with loss scaling
 * (Sec. 3.3, Listing 6).  Nothing in the paper fixes the arithmetic beyond
 * that, so this file writes out the textbook definition:
 *
 *   layout  x[N][C][H][W], w[K][C/g][R][S], y[N][K][P][Q]  (batch, channel,
 *           then spatial; "base axis 1")
 *   P = floor((H + 2*pad_h - dil_h*(R-1) - 1) / stride_h) + 1, same for Q
 *   group of output channel k:  gk = k / (K/g); it reads input channels
 *           gk*(C/g) .. gk*(C/g) + C/g - 1
 *   forward (cross-correlation, no kernel flip, zero padding):
 *     y[n,k,p,q] = alpha * sum_{c'<C/g, r<R, s<S}
 *                  xz[n, gk*C/g + c', p*sh - ph + r*dh, q*sw - pw + s*dw]
 *                  * w[k,c',r,s]
 *     where xz is x extended by zeros outside [0,H) x [0,W).
 *   backward-data: the adjoint of the forward map in x,
 *     dx[n,c,i,j] = alpha * sum over (k in the group of c, r, s, p, q) with
 *                   p*sh - ph + r*dh == i  and  q*sw - pw + s*dw == j
 *                   of dy[n,k,p,q] * w[k, c - gc*C/g, r, s]
 *   backward-weight: the adjoint of the forward map in w, followed by the
 *     loss-scale step of Listing 6 (gradients arrive multiplied by the loss
 *     scale and are divided by it before the update):
 *     dw[k,c',r,s] = beta * dw_old[k,c',r,s] + inv_loss_scale *
 *                    sum_{n,p,q} dy[n,k,p,q] * xz[n, gk*C/g + c', ...]
 *
 * Everything is plain nested loops in double precision, IEEE semantics
 * (build without -ffast-math).  Each full-tensor routine is a loop over
 * output points calling the single-point routine, so a sampled check at
 * large sizes evaluates exactly the same expression.  OpenMP only splits
 * independent output points across threads; every sum is taken serially in
 * the loop order written here.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int64_t n, c, h, w, k, r, s;
    int64_t sh, sw, ph, pw, dh, dw, g;
    int64_t p, q;     /* output spatial size, derived */
    int64_t cg, kg;   /* channels per group (input, output), derived */
} shape_t;

/* Output size from the floor formula.  Returns 0 when the shape is not a
 * valid convolution (non-positive sizes, groups not dividing C and K, or an
 * empty output). */
static int make_shape(shape_t *t, int64_t n, int64_t c, int64_t h, int64_t w,
                      int64_t k, int64_t r, int64_t s, int64_t sh, int64_t sw,
                      int64_t ph, int64_t pw, int64_t dh, int64_t dw, int64_t g)
{
    if (n < 1 || c < 1 || h < 1 || w < 1 || k < 1 || r < 1 || s < 1) return 0;
    if (sh < 1 || sw < 1 || dh < 1 || dw < 1 || ph < 0 || pw < 0 || g < 1) return 0;
    if (c % g != 0 || k % g != 0) return 0;
    int64_t num_h = h + 2 * ph - dh * (r - 1) - 1;
    int64_t num_w = w + 2 * pw - dw * (s - 1) - 1;
    if (num_h < 0 || num_w < 0) return 0;
    t->n = n; t->c = c; t->h = h; t->w = w; t->k = k; t->r = r; t->s = s;
    t->sh = sh; t->sw = sw; t->ph = ph; t->pw = pw; t->dh = dh; t->dw = dw;
    t->g = g;
    t->p = num_h / sh + 1;
    t->q = num_w / sw + 1;
    t->cg = c / g;
    t->kg = k / g;
    return 1;
}

/* x extended by zeros outside the image. */
static double x_at(const shape_t *t, const double *x, int64_t n, int64_t c,
                   int64_t i, int64_t j)
{
    if (i < 0 || i >= t->h || j < 0 || j >= t->w) return 0.0;
    return x[((n * t->c + c) * t->h + i) * t->w + j];
}

/* One forward output point, without alpha. */
static double fwd_point(const shape_t *t, const double *x, const double *w,
                        int64_t n, int64_t k, int64_t p, int64_t q)
{
    int64_t gk = k / t->kg;
    double acc = 0.0;
    for (int64_t cc = 0; cc < t->cg; ++cc)
        for (int64_t r = 0; r < t->r; ++r)
            for (int64_t s = 0; s < t->s; ++s) {
                int64_t i = p * t->sh - t->ph + r * t->dh;
                int64_t j = q * t->sw - t->pw + s * t->dw;
                double xv = x_at(t, x, n, gk * t->cg + cc, i, j);
                double wv = w[((k * t->cg + cc) * t->r + r) * t->s + s];
                acc += xv * wv;
            }
    return acc;
}

/* One backward-data output point, without alpha (gather form).  For each
 * tap (r,s) the forward index equation p*sh - ph + r*dh = i is solved for p;
 * a tap contributes only if the solution is an integer inside [0,P). */
static double dgrad_point(const shape_t *t, const double *dy, const double *w,
                          int64_t n, int64_t c, int64_t i, int64_t j)
{
    int64_t gc = c / t->cg;
    int64_t cc = c - gc * t->cg;
    double acc = 0.0;
    for (int64_t kk = 0; kk < t->kg; ++kk) {
        int64_t k = gc * t->kg + kk;
        for (int64_t r = 0; r < t->r; ++r) {
            int64_t num_p = i + t->ph - r * t->dh;
            if (num_p < 0 || num_p % t->sh != 0) continue;
            int64_t p = num_p / t->sh;
            if (p >= t->p) continue;
            for (int64_t s = 0; s < t->s; ++s) {
                int64_t num_q = j + t->pw - s * t->dw;
                if (num_q < 0 || num_q % t->sw != 0) continue;
                int64_t q = num_q / t->sw;
                if (q >= t->q) continue;
                double dyv = dy[((n * t->k + k) * t->p + p) * t->q + q];
                double wv = w[((k * t->cg + cc) * t->r + r) * t->s + s];
                acc += dyv * wv;
            }
        }
    }
    return acc;
}

/* One backward-weight point: the raw sum over the batch and output pixels,
 * before the loss-scale step. */
static double wgrad_point(const shape_t *t, const double *x, const double *dy,
                          int64_t k, int64_t cc, int64_t r, int64_t s)
{
    int64_t gk = k / t->kg;
    double acc = 0.0;
    for (int64_t n = 0; n < t->n; ++n)
        for (int64_t p = 0; p < t->p; ++p)
            for (int64_t q = 0; q < t->q; ++q) {
                int64_t i = p * t->sh - t->ph + r * t->dh;
                int64_t j = q * t->sw - t->pw + s * t->dw;
                double xv = x_at(t, x, n, gk * t->cg + cc, i, j);
                double dyv = dy[((n * t->k + k) * t->p + p) * t->q + q];
                acc += dyv * xv;
            }
    return acc;
}

#define SHAPE_ARGS int64_t n, int64_t c, int64_t h, int64_t w, int64_t k, \
    int64_t r, int64_t s, int64_t sh, int64_t sw, int64_t ph, int64_t pw, \
    int64_t dh, int64_t dw, int64_t g
#define SHAPE_PASS n, c, h, w, k, r, s, sh, sw, ph, pw, dh, dw, g

/* Output size; returns 0 for an invalid shape. */
int oracle_output_dims(SHAPE_ARGS, int64_t *p, int64_t *q)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    *p = t.p;
    *q = t.q;
    return 1;
}

/* y[N][K][P][Q] = alpha * conv(x, w). */
int oracle_conv_fwd(SHAPE_ARGS, const double *x, const double *wt,
                    double alpha, double *y)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t nn = 0; nn < t.n; ++nn)
        for (int64_t kk = 0; kk < t.k; ++kk)
            for (int64_t p = 0; p < t.p; ++p)
                for (int64_t q = 0; q < t.q; ++q)
                    y[((nn * t.k + kk) * t.p + p) * t.q + q] =
                        alpha * fwd_point(&t, x, wt, nn, kk, p, q);
    return 1;
}

/* dx[N][C][H][W] = alpha * (adjoint of the forward map in x)(dy), gather
 * form. */
int oracle_conv_dgrad(SHAPE_ARGS, const double *dy, const double *wt,
                      double alpha, double *dx)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t nn = 0; nn < t.n; ++nn)
        for (int64_t cc = 0; cc < t.c; ++cc)
            for (int64_t i = 0; i < t.h; ++i)
                for (int64_t j = 0; j < t.w; ++j)
                    dx[((nn * t.c + cc) * t.h + i) * t.w + j] =
                        alpha * dgrad_point(&t, dy, wt, nn, cc, i, j);
    return 1;
}

/* The same backward-data result in scatter form: replay every forward
 * (output point, tap) pair and add dy * w into the input position it read.
 * Independent of the gather form's index inversion; used only as a
 * cross-check of it. */
int oracle_conv_dgrad_scatter(SHAPE_ARGS, const double *dy, const double *wt,
                              double alpha, double *dx)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    int64_t img = t.c * t.h * t.w;
    #pragma omp parallel for schedule(static)
    for (int64_t nn = 0; nn < t.n; ++nn) {
        double *d = dx + nn * img;
        for (int64_t e = 0; e < img; ++e) d[e] = 0.0;
        for (int64_t kk = 0; kk < t.k; ++kk) {
            int64_t gk = kk / t.kg;
            for (int64_t p = 0; p < t.p; ++p)
                for (int64_t q = 0; q < t.q; ++q) {
                    double dyv = dy[((nn * t.k + kk) * t.p + p) * t.q + q];
                    for (int64_t cc = 0; cc < t.cg; ++cc)
                        for (int64_t r = 0; r < t.r; ++r)
                            for (int64_t s = 0; s < t.s; ++s) {
                                int64_t i = p * t.sh - t.ph + r * t.dh;
                                int64_t j = q * t.sw - t.pw + s * t.dw;
                                if (i < 0 || i >= t.h || j < 0 || j >= t.w)
                                    continue;
                                double wv = wt[((kk * t.cg + cc) * t.r + r) * t.s + s];
                                d[((gk * t.cg + cc) * t.h + i) * t.w + j] += dyv * wv;
                            }
                }
        }
        for (int64_t e = 0; e < img; ++e) d[e] *= alpha;
    }
    return 1;
}

/* dw[K][C/g][R][S] = beta * dw + inv_loss_scale * (adjoint in w)(x, dy).
 * beta is 0 or 1 (overwrite or accumulate).  With beta == 0 the old value is
 * not read, so it may hold anything. */
int oracle_conv_wgrad(SHAPE_ARGS, const double *x, const double *dy,
                      double inv_loss_scale, int beta, double *dwt)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t kk = 0; kk < t.k; ++kk)
        for (int64_t cc = 0; cc < t.cg; ++cc)
            for (int64_t r = 0; r < t.r; ++r)
                for (int64_t s = 0; s < t.s; ++s) {
                    int64_t e = ((kk * t.cg + cc) * t.r + r) * t.s + s;
                    double raw = wgrad_point(&t, x, dy, kk, cc, r, s);
                    double old = beta ? dwt[e] : 0.0;
                    dwt[e] = old + inv_loss_scale * raw;
                }
    return 1;
}

/* Sampled forms for large shapes: the same single-point expressions at a
 * caller-chosen list of flat output indices (into the NCHW / KCRS output
 * arrays above). */
int oracle_conv_fwd_points(SHAPE_ARGS, const double *x, const double *wt,
                           double alpha, int64_t npts, const int64_t *idx,
                           double *out)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    #pragma omp parallel for schedule(dynamic, 64)
    for (int64_t e = 0; e < npts; ++e) {
        int64_t f = idx[e];
        int64_t q = f % t.q; f /= t.q;
        int64_t p = f % t.p; f /= t.p;
        int64_t kk = f % t.k; f /= t.k;
        out[e] = alpha * fwd_point(&t, x, wt, f, kk, p, q);
    }
    return 1;
}

int oracle_conv_dgrad_points(SHAPE_ARGS, const double *dy, const double *wt,
                             double alpha, int64_t npts, const int64_t *idx,
                             double *out)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    #pragma omp parallel for schedule(dynamic, 64)
    for (int64_t e = 0; e < npts; ++e) {
        int64_t f = idx[e];
        int64_t j = f % t.w; f /= t.w;
        int64_t i = f % t.h; f /= t.h;
        int64_t cc = f % t.c; f /= t.c;
        out[e] = alpha * dgrad_point(&t, dy, wt, f, cc, i, j);
    }
    return 1;
}

/* Raw weight-gradient sums (no loss-scale step) at chosen KCRS indices. */
int oracle_conv_wgrad_points(SHAPE_ARGS, const double *x, const double *dy,
                             int64_t npts, const int64_t *idx, double *out)
{
    shape_t t;
    if (!make_shape(&t, SHAPE_PASS)) return 0;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t e = 0; e < npts; ++e) {
        int64_t f = idx[e];
        int64_t s = f % t.s; f /= t.s;
        int64_t r = f % t.r; f /= t.r;
        int64_t cc = f % t.cg; f /= t.cg;
        out[e] = wgrad_point(&t, x, dy, f, cc, r, s);
    }
    return 1;
}

/* Listing 6's check_inf_or_nan_grad over one gradient array: 1 when any
 * element is an infinity or a NaN. */
int oracle_any_nonfinite(const double *v, int64_t len)
{
    for (int64_t e = 0; e < len; ++e)
        if (!isfinite(v[e])) return 1;
    return 0;
}

/* Thread count used by the OpenMP loops above (1 when built without
 * OpenMP). */
void oracle_set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

int oracle_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
