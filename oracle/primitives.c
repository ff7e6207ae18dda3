/*
 * oracle/primitives.c -- CPU oracle for the 3D-ResAttNet training step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * includes this file; only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark use it.  It shares no code, header or table with the HIP
 * path.
 *
 * Every routine is the plain definition of the operation, in double precision,
 * written as nested loops.  The loop order puts the output positions innermost
 * so that the compiler can vectorise them; each output still receives exactly
 * the terms of the defining sum (summation order is the only freedom taken).
 *
 * Operations (all tensors contiguous NCDHW, weights [Co][Ci][k][k][k]):
 *   - 3D convolution forward / input gradient / weight gradient.  The paper
 *     builds its conv blocks from 3x3x3 convolutions (use-case section, the
 *     conv block description) and prices a layer at
 *     O(C_o C_i T H W K_T K_H K_W) (same section): these loops are that sum.
 *   - 3D max pooling with a first-maximum argmax, and its gradient.
 *   - trilinear resampling to an explicit target size (half-pixel centres,
 *     border clamp), and its exact transpose.
 * The pooling / resampling steps are the soft-mask branch of the residual
 * attention block, which the paper names but does not specify; the reading
 * used (max pool 3^3 stride 2 pad 1, trilinear up to the pre-pool size) is
 * the one recorded in the design notes of the repository.
 */
#include <stdint.h>
#include <stddef.h>
#include <math.h>

#define IDX5(n, c, d, h, w, C, D, H, W) \
    ((((((int64_t)(n) * (C) + (c)) * (D) + (d)) * (H) + (h)) * (W) + (w)))

int orc_out_size(int in, int k, int s, int p) { return (in + 2 * p - k) / s + 1; }

/* Output positions o in [0, out) whose input tap position o*s - p + t lies in
 * [0, in): returns the half-open range [*lo, *hi). */
static void tap_range(int t, int s, int p, int in, int out, int* lo, int* hi)
{
    int a = 0, b = out;
    /* need o*s - p + t >= 0  ->  o >= ceil((p - t) / s) */
    int num = p - t;
    if (num > 0) a = (num + s - 1) / s;
    /* need o*s - p + t <= in - 1  ->  o <= floor((in - 1 + p - t) / s) */
    int num2 = in - 1 + p - t;
    if (num2 < 0) b = 0;
    else if (num2 / s + 1 < b) b = num2 / s + 1;
    if (a > b) a = b;
    *lo = a;
    *hi = b;
}

/* y[n,co,o] = bias[co] + sum_{ci,kd,kh,kw} w[co,ci,kd,kh,kw] * x[n,ci,o*s-p+k]
 * with zero padding outside the input volume. */
void orc_conv3d_fwd(int N, int Ci, int Co, int D, int H, int W, int k, int s, int p,
                    const double* x, const double* w, const double* bias, double* y)
{
    const int Do = orc_out_size(D, k, s, p), Ho = orc_out_size(H, k, s, p),
              Wo = orc_out_size(W, k, s, p);
    const int64_t vo = (int64_t)Do * Ho * Wo;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int n = 0; n < N; ++n)
        for (int co = 0; co < Co; ++co) {
            double* yp = y + ((int64_t)n * Co + co) * vo;
            const double b0 = bias ? bias[co] : 0.0;
            for (int64_t i = 0; i < vo; ++i) yp[i] = b0;
            for (int ci = 0; ci < Ci; ++ci) {
                const double* xp = x + ((int64_t)n * Ci + ci) * D * H * W;
                for (int kd = 0; kd < k; ++kd)
                    for (int kh = 0; kh < k; ++kh)
                        for (int kw = 0; kw < k; ++kw) {
                            const double wv =
                                w[((((int64_t)co * Ci + ci) * k + kd) * k + kh) * k + kw];
                            int d0, d1, h0, h1, w0, w1;
                            tap_range(kd, s, p, D, Do, &d0, &d1);
                            tap_range(kh, s, p, H, Ho, &h0, &h1);
                            tap_range(kw, s, p, W, Wo, &w0, &w1);
                            for (int od = d0; od < d1; ++od) {
                                const int id = od * s - p + kd;
                                for (int oh = h0; oh < h1; ++oh) {
                                    const int ih = oh * s - p + kh;
                                    double* yr = yp + ((int64_t)od * Ho + oh) * Wo;
                                    const double* xr = xp + ((int64_t)id * H + ih) * W;
                                    for (int ow = w0; ow < w1; ++ow)
                                        yr[ow] += wv * xr[ow * s - p + kw];
                                }
                            }
                        }
            }
        }
}

/* Input gradient, written from its own definition (not as a flipped forward):
 * dx[n,ci,i] = sum over (co, t) with (i + p - t) divisible by s and
 * 0 <= (i + p - t)/s < out, of w[co,ci,t] * dy[n,co,(i + p - t)/s]
 * (per axis).  If accumulate != 0 the result is added to dx. */
void orc_conv3d_dgrad(int N, int Ci, int Co, int D, int H, int W, int k, int s, int p,
                      const double* dy, const double* w, double* dx, int accumulate)
{
    const int Do = orc_out_size(D, k, s, p), Ho = orc_out_size(H, k, s, p),
              Wo = orc_out_size(W, k, s, p);
    const int64_t vi = (int64_t)D * H * W, vo = (int64_t)Do * Ho * Wo;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int n = 0; n < N; ++n)
        for (int ci = 0; ci < Ci; ++ci) {
            double* dxp = dx + ((int64_t)n * Ci + ci) * vi;
            if (!accumulate)
                for (int64_t i = 0; i < vi; ++i) dxp[i] = 0.0;
            for (int co = 0; co < Co; ++co) {
                const double* dyp = dy + ((int64_t)n * Co + co) * vo;
                for (int kd = 0; kd < k; ++kd)
                    for (int kh = 0; kh < k; ++kh)
                        for (int kw = 0; kw < k; ++kw) {
                            const double wv =
                                w[((((int64_t)co * Ci + ci) * k + kd) * k + kh) * k + kw];
                            for (int id = 0; id < D; ++id) {
                                const int nd = id + p - kd;
                                if (nd < 0 || nd % s != 0 || nd / s >= Do) continue;
                                const int od = nd / s;
                                for (int ih = 0; ih < H; ++ih) {
                                    const int nh = ih + p - kh;
                                    if (nh < 0 || nh % s != 0 || nh / s >= Ho) continue;
                                    const int oh = nh / s;
                                    double* dxr = dxp + ((int64_t)id * H + ih) * W;
                                    const double* dyr = dyp + ((int64_t)od * Ho + oh) * Wo;
                                    if (s == 1) {
                                        /* ow = iw + p - kw must lie in [0, Wo) */
                                        int lo = kw - p, hi = kw - p + Wo;
                                        if (lo < 0) lo = 0;
                                        if (hi > W) hi = W;
                                        for (int iw = lo; iw < hi; ++iw)
                                            dxr[iw] += wv * dyr[iw + p - kw];
                                    } else {
                                        for (int iw = 0; iw < W; ++iw) {
                                            const int nw = iw + p - kw;
                                            if (nw < 0 || nw % s != 0 || nw / s >= Wo) continue;
                                            dxr[iw] += wv * dyr[nw / s];
                                        }
                                    }
                                }
                            }
                        }
            }
        }
}

/* dw[co,ci,t] = sum_n sum_o dy[n,co,o] * x[n,ci,o*s-p+t];  db[co] = sum_n sum_o dy[n,co,o].
 * If accumulate != 0 the results are added to dw / db. */
void orc_conv3d_wgrad(int N, int Ci, int Co, int D, int H, int W, int k, int s, int p,
                      const double* x, const double* dy, double* dw, double* db, int accumulate)
{
    const int Do = orc_out_size(D, k, s, p), Ho = orc_out_size(H, k, s, p),
              Wo = orc_out_size(W, k, s, p);
    const int64_t vi = (int64_t)D * H * W, vo = (int64_t)Do * Ho * Wo;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int co = 0; co < Co; ++co)
        for (int ci = 0; ci < Ci; ++ci)
            for (int kd = 0; kd < k; ++kd)
                for (int kh = 0; kh < k; ++kh)
                    for (int kw = 0; kw < k; ++kw) {
                        int d0, d1, h0, h1, w0, w1;
                        tap_range(kd, s, p, D, Do, &d0, &d1);
                        tap_range(kh, s, p, H, Ho, &h0, &h1);
                        tap_range(kw, s, p, W, Wo, &w0, &w1);
                        double acc = 0.0;
                        for (int n = 0; n < N; ++n) {
                            const double* xp = x + ((int64_t)n * Ci + ci) * vi;
                            const double* dyp = dy + ((int64_t)n * Co + co) * vo;
                            for (int od = d0; od < d1; ++od) {
                                const int id = od * s - p + kd;
                                for (int oh = h0; oh < h1; ++oh) {
                                    const int ih = oh * s - p + kh;
                                    const double* dyr = dyp + ((int64_t)od * Ho + oh) * Wo;
                                    const double* xr = xp + ((int64_t)id * H + ih) * W;
                                    for (int ow = w0; ow < w1; ++ow)
                                        acc += dyr[ow] * xr[ow * s - p + kw];
                                }
                            }
                        }
                        double* dst =
                            &dw[((((int64_t)co * Ci + ci) * k + kd) * k + kh) * k + kw];
                        *dst = accumulate ? *dst + acc : acc;
                    }
    if (db) {
        for (int co = 0; co < Co; ++co) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n) {
                const double* dyp = dy + ((int64_t)n * Co + co) * vo;
                for (int64_t i = 0; i < vo; ++i) acc += dyp[i];
            }
            db[co] = accumulate ? db[co] + acc : acc;
        }
    }
}

/* Max pooling, window k^3, stride s, padding p (padded taps never win).
 * The argmax is the window offset (kd*k + kh)*k + kw of the FIRST maximum in
 * (kd, kh, kw) scan order: a later tap replaces the current best only if it is
 * strictly greater. */
void orc_maxpool3d_fwd(int N, int C, int D, int H, int W, int k, int s, int p,
                       const double* x, double* y, int32_t* argmax)
{
    const int Do = orc_out_size(D, k, s, p), Ho = orc_out_size(H, k, s, p),
              Wo = orc_out_size(W, k, s, p);
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c)
            for (int od = 0; od < Do; ++od)
                for (int oh = 0; oh < Ho; ++oh)
                    for (int ow = 0; ow < Wo; ++ow) {
                        double best = -INFINITY;
                        int arg = -1;
                        for (int kd = 0; kd < k; ++kd)
                            for (int kh = 0; kh < k; ++kh)
                                for (int kw = 0; kw < k; ++kw) {
                                    const int id = od * s - p + kd, ih = oh * s - p + kh,
                                              iw = ow * s - p + kw;
                                    if (id < 0 || id >= D || ih < 0 || ih >= H || iw < 0 ||
                                        iw >= W)
                                        continue;
                                    const double v = x[IDX5(n, c, id, ih, iw, C, D, H, W)];
                                    if (arg < 0 || v > best) {
                                        best = v;
                                        arg = (kd * k + kh) * k + kw;
                                    }
                                }
                        const int64_t o = IDX5(n, c, od, oh, ow, C, Do, Ho, Wo);
                        y[o] = best;
                        argmax[o] = arg;
                    }
}

/* Gradient of max pooling: every output sends its gradient to the input voxel
 * its argmax names.  If accumulate != 0 the result is added to dx. */
void orc_maxpool3d_bwd(int N, int C, int D, int H, int W, int k, int s, int p,
                       const double* dy, const int32_t* argmax, double* dx, int accumulate)
{
    const int Do = orc_out_size(D, k, s, p), Ho = orc_out_size(H, k, s, p),
              Wo = orc_out_size(W, k, s, p);
    const int64_t vi = (int64_t)D * H * W;
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c) {
            double* dxp = dx + ((int64_t)n * C + c) * vi;
            if (!accumulate)
                for (int64_t i = 0; i < vi; ++i) dxp[i] = 0.0;
            for (int od = 0; od < Do; ++od)
                for (int oh = 0; oh < Ho; ++oh)
                    for (int ow = 0; ow < Wo; ++ow) {
                        const int64_t o = IDX5(n, c, od, oh, ow, C, Do, Ho, Wo);
                        const int a = argmax[o];
                        const int kd = a / (k * k), kh = (a / k) % k, kw = a % k;
                        const int id = od * s - p + kd, ih = oh * s - p + kh,
                                  iw = ow * s - p + kw;
                        dxp[((int64_t)id * H + ih) * W + iw] += dy[o];
                    }
        }
}

/* Source coordinate of output index o when resampling an axis of length `in`
 * to length `out` with half-pixel centres: src = (o + 1/2) * in/out - 1/2,
 * clamped below at 0; i0 = floor(src), i1 = min(i0 + 1, in - 1),
 * lambda = src - i0 (weight of i1). */
static void lin_src(int o, int in, int out, int* i0, int* i1, double* lam)
{
    double src = ((double)o + 0.5) * ((double)in / (double)out) - 0.5;
    if (src < 0.0) src = 0.0;
    int a = (int)floor(src);
    if (a > in - 1) a = in - 1;
    *i0 = a;
    *i1 = a + 1 < in ? a + 1 : in - 1;
    *lam = src - (double)a;
}

/* Trilinear resampling of each (n, c) volume from Di x Hi x Wi to Do x Ho x Wo:
 * y = sum over the 8 corners of the product of the per-axis linear weights. */
void orc_trilinear_fwd(int N, int C, int Di, int Hi, int Wi, int Do, int Ho, int Wo,
                       const double* x, double* y)
{
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c) {
            const double* xp = x + ((int64_t)n * C + c) * Di * Hi * Wi;
            double* yp = y + ((int64_t)n * C + c) * Do * Ho * Wo;
            for (int od = 0; od < Do; ++od) {
                int d0, d1; double ld;
                lin_src(od, Di, Do, &d0, &d1, &ld);
                for (int oh = 0; oh < Ho; ++oh) {
                    int h0, h1; double lh;
                    lin_src(oh, Hi, Ho, &h0, &h1, &lh);
                    for (int ow = 0; ow < Wo; ++ow) {
                        int w0, w1; double lw;
                        lin_src(ow, Wi, Wo, &w0, &w1, &lw);
                        const int dd[2] = {d0, d1}, hh[2] = {h0, h1}, ww[2] = {w0, w1};
                        const double wd[2] = {1.0 - ld, ld}, wh[2] = {1.0 - lh, lh},
                                     wwt[2] = {1.0 - lw, lw};
                        double acc = 0.0;
                        for (int a = 0; a < 2; ++a)
                            for (int b = 0; b < 2; ++b)
                                for (int e = 0; e < 2; ++e)
                                    acc += wd[a] * wh[b] * wwt[e] *
                                           xp[((int64_t)dd[a] * Hi + hh[b]) * Wi + ww[e]];
                        yp[((int64_t)od * Ho + oh) * Wo + ow] = acc;
                    }
                }
            }
        }
}

/* Transpose of orc_trilinear_fwd: each output gradient is spread over its 8
 * source corners with the same weights.  If accumulate != 0, added to dx. */
void orc_trilinear_bwd(int N, int C, int Di, int Hi, int Wi, int Do, int Ho, int Wo,
                       const double* dy, double* dx, int accumulate)
{
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c) {
            double* dxp = dx + ((int64_t)n * C + c) * Di * Hi * Wi;
            const double* dyp = dy + ((int64_t)n * C + c) * Do * Ho * Wo;
            if (!accumulate)
                for (int64_t i = 0; i < (int64_t)Di * Hi * Wi; ++i) dxp[i] = 0.0;
            for (int od = 0; od < Do; ++od) {
                int d0, d1; double ld;
                lin_src(od, Di, Do, &d0, &d1, &ld);
                for (int oh = 0; oh < Ho; ++oh) {
                    int h0, h1; double lh;
                    lin_src(oh, Hi, Ho, &h0, &h1, &lh);
                    for (int ow = 0; ow < Wo; ++ow) {
                        int w0, w1; double lw;
                        lin_src(ow, Wi, Wo, &w0, &w1, &lw);
                        const int dd[2] = {d0, d1}, hh[2] = {h0, h1}, ww[2] = {w0, w1};
                        const double wd[2] = {1.0 - ld, ld}, wh[2] = {1.0 - lh, lh},
                                     wwt[2] = {1.0 - lw, lw};
                        const double g = dyp[((int64_t)od * Ho + oh) * Wo + ow];
                        for (int a = 0; a < 2; ++a)
                            for (int b = 0; b < 2; ++b)
                                for (int e = 0; e < 2; ++e)
                                    dxp[((int64_t)dd[a] * Hi + hh[b]) * Wi + ww[e]] +=
                                        wd[a] * wh[b] * wwt[e] * g;
                    }
                }
            }
        }
}

/* ---- Sampled outputs (for checks at sizes where the full oracle is too slow).
 * Each routine evaluates the same defining sums as above at a list of points.
 * pts holds npts records of 5 ints. */

/* y at points (n, co, od, oh, ow). */
void orc_conv3d_fwd_points(int N, int Ci, int Co, int D, int H, int W, int k, int s, int p,
                           const double* x, const double* w, const double* bias,
                           int npts, const int32_t* pts, double* out)
{
    (void)N; (void)Co;
#pragma omp parallel for schedule(dynamic)
    for (int q = 0; q < npts; ++q) {
        const int n = pts[5 * q], co = pts[5 * q + 1], od = pts[5 * q + 2],
                  oh = pts[5 * q + 3], ow = pts[5 * q + 4];
        double acc = bias ? bias[co] : 0.0;
        for (int ci = 0; ci < Ci; ++ci)
            for (int kd = 0; kd < k; ++kd)
                for (int kh = 0; kh < k; ++kh)
                    for (int kw = 0; kw < k; ++kw) {
                        const int id = od * s - p + kd, ih = oh * s - p + kh,
                                  iw = ow * s - p + kw;
                        if (id < 0 || id >= D || ih < 0 || ih >= H || iw < 0 || iw >= W)
                            continue;
                        acc += w[((((int64_t)co * Ci + ci) * k + kd) * k + kh) * k + kw] *
                               x[IDX5(n, ci, id, ih, iw, Ci, D, H, W)];
                    }
        out[q] = acc;
    }
}

/* dx at points (n, ci, id, ih, iw). */
void orc_conv3d_dgrad_points(int N, int Ci, int Co, int D, int H, int W, int k, int s, int p,
                             const double* dy, const double* w,
                             int npts, const int32_t* pts, double* out)
{
    (void)N;
    const int Do = orc_out_size(D, k, s, p), Ho = orc_out_size(H, k, s, p),
              Wo = orc_out_size(W, k, s, p);
#pragma omp parallel for schedule(dynamic)
    for (int q = 0; q < npts; ++q) {
        const int n = pts[5 * q], ci = pts[5 * q + 1], id = pts[5 * q + 2],
                  ih = pts[5 * q + 3], iw = pts[5 * q + 4];
        double acc = 0.0;
        for (int co = 0; co < Co; ++co)
            for (int kd = 0; kd < k; ++kd)
                for (int kh = 0; kh < k; ++kh)
                    for (int kw = 0; kw < k; ++kw) {
                        const int nd = id + p - kd, nh = ih + p - kh, nw = iw + p - kw;
                        if (nd < 0 || nh < 0 || nw < 0) continue;
                        if (nd % s || nh % s || nw % s) continue;
                        const int od = nd / s, oh = nh / s, ow = nw / s;
                        if (od >= Do || oh >= Ho || ow >= Wo) continue;
                        acc += w[((((int64_t)co * Ci + ci) * k + kd) * k + kh) * k + kw] *
                               dy[IDX5(n, co, od, oh, ow, Co, Do, Ho, Wo)];
                    }
        out[q] = acc;
    }
}

/* dw at points (co, ci, kd, kh, kw); the sum runs over the whole batch. */
void orc_conv3d_wgrad_points(int N, int Ci, int Co, int D, int H, int W, int k, int s, int p,
                             const double* x, const double* dy,
                             int npts, const int32_t* pts, double* out)
{
    const int Do = orc_out_size(D, k, s, p), Ho = orc_out_size(H, k, s, p),
              Wo = orc_out_size(W, k, s, p);
#pragma omp parallel for schedule(dynamic)
    for (int q = 0; q < npts; ++q) {
        const int co = pts[5 * q], ci = pts[5 * q + 1], kd = pts[5 * q + 2],
                  kh = pts[5 * q + 3], kw = pts[5 * q + 4];
        double acc = 0.0;
        for (int n = 0; n < N; ++n)
            for (int od = 0; od < Do; ++od) {
                const int id = od * s - p + kd;
                if (id < 0 || id >= D) continue;
                for (int oh = 0; oh < Ho; ++oh) {
                    const int ih = oh * s - p + kh;
                    if (ih < 0 || ih >= H) continue;
                    for (int ow = 0; ow < Wo; ++ow) {
                        const int iw = ow * s - p + kw;
                        if (iw < 0 || iw >= W) continue;
                        acc += dy[IDX5(n, co, od, oh, ow, Co, Do, Ho, Wo)] *
                               x[IDX5(n, ci, id, ih, iw, Ci, D, H, W)];
                    }
                }
            }
        out[q] = acc;
    }
}

/* Threads the oracle's parallel loops use. */
#include <omp.h>
int orc_num_threads(void) { return omp_get_max_threads(); }
