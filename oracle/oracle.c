/*
 * Plain CPU oracle for the three training passes of a convolution layer,
 * and for the forward and backward passes of a pooling layer (at the end).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header or constant with the HIP
 * library.
 *
 * What it computes (swCaffe, Sec. IV-B "Convolutional Layer" and Table II):
 * a convolution layer maps an input tensor x[N][C][H][W] and a filter bank
 * w[K][C/G][R][S] (plus bias b[K]) to y[N][K][P][Q].  Sec. IV-B writes the
 * forward pass as im2col followed by a GEMM whose common dimension is
 * (filter height x filter width x input channels); the backward pass moves
 * data back with col2im.  Table II names the three passes: forward,
 * weight_diff backward and in_diff backward.  Padding is zero padding
 * (Sec. IV-B, implicit-GEMM paragraph), tensors are (batch, channel, row,
 * column) and filters (out-channel, in-channel, row, column)
 * (Sec. IV-C, explicit-plan layouts).
 *
 * Readings where the paper is silent (all follow Caffe's convolution layer):
 *   - output size P = floor((H + 2 pad - R) / stride) + 1 (Sec. IV-B prints
 *     (Ci - K)/S + 1 without padding or rounding);
 *   - cross-correlation (the im2col matrix multiplies the unflipped filter);
 *   - groups split input channels and filters into G contiguous blocks;
 *   - bias is one scalar per output channel; db sums dy over n, p, q;
 *   - outputs are overwritten, not accumulated.
 *
 * Arithmetic: every input arrives as double (the canonical fp32 inputs
 * convert exactly), every sum is accumulated in double in loop order.
 * Alongside each value the oracle returns the sum of the absolute values of
 * every product that entered it (plus |b| for y); that is the per-element
 * scale of the tolerance.
 *
 * Two forms of each backward pass are given on purpose:
 *   - the full-tensor functions run the forward index loop and scatter-add
 *     into dx / dw (the col2im adjoint of Sec. IV-B);
 *   - the *_at functions gather one element straight from its definition.
 * The tests check the two forms against each other.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -fPIC -shared (no fast-math).
 */
#include <stddef.h>
#include <stdint.h>
#include <math.h>
#include <omp.h>

typedef int64_t i64;

/* Output extent along one axis: zero padding on both sides, floor rounding.
 * Returns < 1 when the window does not fit. */
int oracle_out_size(int in, int filt, int stride, int pad)
{
    i64 span = (i64)in + 2 * (i64)pad - (i64)filt;
    if (stride < 1 || span < 0)
        return 0;
    return (int)(span / stride + 1);
}

int oracle_num_threads(void)
{
    return omp_get_max_threads();
}

/* x at (n, c, h, w) with zero padding: out-of-range coordinates read 0. */
static double x_at(const double *x, int C, int H, int W, int n, int c, i64 h, i64 w)
{
    if (h < 0 || h >= H || w < 0 || w >= W)
        return 0.0;
    return x[(((i64)n * C + c) * H + h) * W + w];
}

/* ------------------------------------------------------------------ */
/* Forward: y[n,k,p,q] = b[k] + sum_{c<C/G, r, s} x[n, g*C/G + c,     */
/*          p*st - pad + r, q*st - pad + s] * w[k, c, r, s],          */
/* with g = k / (K/G).  b may be NULL (no bias).                       */
/* ------------------------------------------------------------------ */
void oracle_conv_fwd(int N, int C, int H, int W, int K, int R, int S,
                     int stride, int pad, int group,
                     const double *x, const double *w, const double *b,
                     double *y, double *ay)
{
    int P = oracle_out_size(H, R, stride, pad);
    int Q = oracle_out_size(W, S, stride, pad);
    int Cg = C / group, Kg = K / group;
    i64 nk;
#pragma omp parallel for schedule(dynamic)
    for (nk = 0; nk < (i64)N * K; nk++) {
        int n = (int)(nk / K), k = (int)(nk % K);
        int g = k / Kg;
        for (int p = 0; p < P; p++)
            for (int q = 0; q < Q; q++) {
                double acc = 0.0, aacc = 0.0;
                if (b) {
                    acc = b[k];
                    aacc = fabs(b[k]);
                }
                for (int c = 0; c < Cg; c++)
                    for (int r = 0; r < R; r++)
                        for (int s = 0; s < S; s++) {
                            double xv = x_at(x, C, H, W, n, g * Cg + c,
                                             (i64)p * stride - pad + r,
                                             (i64)q * stride - pad + s);
                            double wv = w[(((i64)k * Cg + c) * R + r) * S + s];
                            acc += xv * wv;
                            aacc += fabs(xv * wv);
                        }
                i64 o = (((i64)n * K + k) * P + p) * Q + q;
                y[o] = acc;
                if (ay)
                    ay[o] = aacc;
            }
    }
}

/* ------------------------------------------------------------------ */
/* Backward-data, scatter form (col2im adjoint of the forward loop):  */
/* for every forward product x[n,c',h,w] * w[k,c,r,s] that reached    */
/* y[n,k,p,q], add dy[n,k,p,q] * w[k,c,r,s] into dx[n,c',h,w].         */
/* Pixels no window covers stay exactly 0.                            */
/* One thread owns one (n, input channel) plane, so there is no race. */
/* ------------------------------------------------------------------ */
void oracle_conv_bwd_data(int N, int C, int H, int W, int K, int R, int S,
                          int stride, int pad, int group,
                          const double *dy, const double *w,
                          double *dx, double *adx)
{
    int P = oracle_out_size(H, R, stride, pad);
    int Q = oracle_out_size(W, S, stride, pad);
    int Cg = C / group, Kg = K / group;
    i64 nc;
#pragma omp parallel for schedule(dynamic)
    for (nc = 0; nc < (i64)N * C; nc++) {
        int n = (int)(nc / C), cc = (int)(nc % C);
        int g = cc / Cg, c = cc % Cg;
        double *plane = dx + nc * H * W;
        double *aplane = adx ? adx + nc * H * W : NULL;
        for (i64 i = 0; i < (i64)H * W; i++) {
            plane[i] = 0.0;
            if (aplane)
                aplane[i] = 0.0;
        }
        for (int k = g * Kg; k < (g + 1) * Kg; k++)
            for (int p = 0; p < P; p++)
                for (int q = 0; q < Q; q++) {
                    double d = dy[(((i64)n * K + k) * P + p) * Q + q];
                    for (int r = 0; r < R; r++)
                        for (int s = 0; s < S; s++) {
                            i64 h = (i64)p * stride - pad + r;
                            i64 wc = (i64)q * stride - pad + s;
                            if (h < 0 || h >= H || wc < 0 || wc >= W)
                                continue;
                            double prod = d * w[(((i64)k * Cg + c) * R + r) * S + s];
                            plane[h * W + wc] += prod;
                            if (aplane)
                                aplane[h * W + wc] += fabs(prod);
                        }
                }
    }
}

/* ------------------------------------------------------------------ */
/* Backward-weight, scatter form: for every forward product, add      */
/* dy[n,k,p,q] * x[n,c',h,w] into dw[k,c,r,s]; db[k] sums dy[n,k,:,:]. */
/* One thread owns one output channel k.  db / adb may be NULL.       */
/* ------------------------------------------------------------------ */
void oracle_conv_bwd_weight(int N, int C, int H, int W, int K, int R, int S,
                            int stride, int pad, int group,
                            const double *x, const double *dy,
                            double *dw, double *adw, double *db, double *adb)
{
    int P = oracle_out_size(H, R, stride, pad);
    int Q = oracle_out_size(W, S, stride, pad);
    int Cg = C / group, Kg = K / group;
    int k;
#pragma omp parallel for schedule(dynamic)
    for (k = 0; k < K; k++) {
        int g = k / Kg;
        double *dwk = dw + (i64)k * Cg * R * S;
        double *adwk = adw ? adw + (i64)k * Cg * R * S : NULL;
        for (i64 i = 0; i < (i64)Cg * R * S; i++) {
            dwk[i] = 0.0;
            if (adwk)
                adwk[i] = 0.0;
        }
        double bsum = 0.0, absum = 0.0;
        for (int n = 0; n < N; n++)
            for (int p = 0; p < P; p++)
                for (int q = 0; q < Q; q++) {
                    double d = dy[(((i64)n * K + k) * P + p) * Q + q];
                    bsum += d;
                    absum += fabs(d);
                    for (int c = 0; c < Cg; c++)
                        for (int r = 0; r < R; r++)
                            for (int s = 0; s < S; s++) {
                                double xv = x_at(x, C, H, W, n, g * Cg + c,
                                                 (i64)p * stride - pad + r,
                                                 (i64)q * stride - pad + s);
                                i64 o = ((i64)c * R + r) * S + s;
                                dwk[o] += d * xv;
                                if (adwk)
                                    adwk[o] += fabs(d * xv);
                            }
                }
        if (db)
            db[k] = bsum;
        if (adb)
            adb[k] = absum;
    }
}

/* ------------------------------------------------------------------ */
/* Per-element gather forms, for sampling outputs of full-size layers. */
/* Each takes a list of flat output indices and writes one value and  */
/* one abs-sum per index.  Parallel over the list.                    */
/* ------------------------------------------------------------------ */

/* y at flat index into [N][K][P][Q]. */
void oracle_conv_fwd_at(int N, int C, int H, int W, int K, int R, int S,
                        int stride, int pad, int group,
                        const double *x, const double *w, const double *b,
                        const i64 *idx, i64 count, double *val, double *aval)
{
    int P = oracle_out_size(H, R, stride, pad);
    int Q = oracle_out_size(W, S, stride, pad);
    int Cg = C / group, Kg = K / group;
    i64 t;
    (void)N;
#pragma omp parallel for schedule(dynamic)
    for (t = 0; t < count; t++) {
        i64 o = idx[t];
        int q = (int)(o % Q);
        int p = (int)((o / Q) % P);
        int k = (int)((o / ((i64)Q * P)) % K);
        int n = (int)(o / ((i64)Q * P * K));
        int g = k / Kg;
        double acc = b ? b[k] : 0.0, aacc = b ? fabs(b[k]) : 0.0;
        for (int c = 0; c < Cg; c++)
            for (int r = 0; r < R; r++)
                for (int s = 0; s < S; s++) {
                    double xv = x_at(x, C, H, W, n, g * Cg + c,
                                     (i64)p * stride - pad + r, (i64)q * stride - pad + s);
                    double wv = w[(((i64)k * Cg + c) * R + r) * S + s];
                    acc += xv * wv;
                    aacc += fabs(xv * wv);
                }
        val[t] = acc;
        aval[t] = aacc;
    }
}

/* dx at flat index into [N][C][H][W]: sum over the filters of the
 * pixel's group and the taps (r, s) whose window position p, q is an
 * integer inside the output, i.e. h + pad - r a non-negative multiple
 * of the stride with quotient below P (same for w, s, Q). */
void oracle_conv_bwd_data_at(int N, int C, int H, int W, int K, int R, int S,
                             int stride, int pad, int group,
                             const double *dy, const double *w,
                             const i64 *idx, i64 count, double *val, double *aval)
{
    int P = oracle_out_size(H, R, stride, pad);
    int Q = oracle_out_size(W, S, stride, pad);
    int Cg = C / group, Kg = K / group;
    i64 t;
    (void)N;
#pragma omp parallel for schedule(dynamic)
    for (t = 0; t < count; t++) {
        i64 o = idx[t];
        int wc = (int)(o % W);
        int h = (int)((o / W) % H);
        int cc = (int)((o / ((i64)W * H)) % C);
        int n = (int)(o / ((i64)W * H * C));
        int g = cc / Cg, c = cc % Cg;
        double acc = 0.0, aacc = 0.0;
        for (int k = g * Kg; k < (g + 1) * Kg; k++)
            for (int r = 0; r < R; r++)
                for (int s = 0; s < S; s++) {
                    i64 ph = (i64)h + pad - r, qw = (i64)wc + pad - s;
                    if (ph < 0 || qw < 0 || ph % stride || qw % stride)
                        continue;
                    ph /= stride;
                    qw /= stride;
                    if (ph >= P || qw >= Q)
                        continue;
                    double prod = dy[(((i64)n * K + k) * P + ph) * Q + qw] *
                                  w[(((i64)k * Cg + c) * R + r) * S + s];
                    acc += prod;
                    aacc += fabs(prod);
                }
        val[t] = acc;
        aval[t] = aacc;
    }
}

/* dw at flat index into [K][C/G][R][S]. */
void oracle_conv_bwd_weight_at(int N, int C, int H, int W, int K, int R, int S,
                               int stride, int pad, int group,
                               const double *x, const double *dy,
                               const i64 *idx, i64 count, double *val, double *aval)
{
    int P = oracle_out_size(H, R, stride, pad);
    int Q = oracle_out_size(W, S, stride, pad);
    int Cg = C / group, Kg = K / group;
    i64 t;
#pragma omp parallel for schedule(dynamic)
    for (t = 0; t < count; t++) {
        i64 o = idx[t];
        int s = (int)(o % S);
        int r = (int)((o / S) % R);
        int c = (int)((o / ((i64)S * R)) % Cg);
        int k = (int)(o / ((i64)S * R * Cg));
        int g = k / Kg;
        double acc = 0.0, aacc = 0.0;
        for (int n = 0; n < N; n++)
            for (int p = 0; p < P; p++)
                for (int q = 0; q < Q; q++) {
                    double prod = dy[(((i64)n * K + k) * P + p) * Q + q] *
                                  x_at(x, C, H, W, n, g * Cg + c,
                                       (i64)p * stride - pad + r, (i64)q * stride - pad + s);
                    acc += prod;
                    aacc += fabs(prod);
                }
        val[t] = acc;
        aval[t] = aacc;
    }
}

/* db alone: db[k] = sum over n, p, q of dy[n,k,p,q] (with its abs-sum),
 * for sampling the bias gradient of full-size layers. */
void oracle_bias_grad(int N, int K, int P, int Q, const double *dy,
                      double *db, double *adb)
{
    int k;
#pragma omp parallel for schedule(static)
    for (k = 0; k < K; k++) {
        double acc = 0.0, aacc = 0.0;
        for (int n = 0; n < N; n++)
            for (i64 i = 0; i < (i64)P * Q; i++) {
                double d = dy[((i64)n * K + k) * P * Q + i];
                acc += d;
                aacc += fabs(d);
            }
        db[k] = acc;
        adb[k] = aacc;
    }
}

/* ------------------------------------------------------------------ */
/* Pooling (Sec. IV-D): each output is the maximum or the average of   */
/* one window of its input plane.  The paper's layer tiles the image   */
/* into non-overlapping K x K windows; the general Caffe form below    */
/* (window R x S, stride, zero padding) contains that case             */
/* (R = S = stride, pad = 0).  Readings (Caffe's pooling layer):       */
/*   - output size ceil((H + 2 pad - R) / stride) + 1, less one when    */
/*     pad > 0 and the last window would start at or past H + pad; a    */
/*     size whose last window would hold no image element (possible     */
/*     without padding when stride > R) is refused (0): a window must   */
/*     hold at least one element;                                       */
/*   - max: over the window's elements inside the image (padding never  */
/*     wins); the argmax is the first maximum in row-major order, kept  */
/*     as the index h * W + w within the plane;                         */
/*   - avg: the sum over the window's elements inside the image divided */
/*     by the window's area clipped to the padded image [-pad, H + pad) */
/*     (padding counts as zeros, the overhang past it does not).        */
/* The backward pass routes dy back along the same definition, in the   */
/* scatter form: max adds dy to its argmax, avg adds dy / area to every */
/* element of its window inside the image.                              */
/* ------------------------------------------------------------------ */
int oracle_pool_out_size(int in, int filt, int stride, int pad)
{
    i64 span = (i64)in + 2 * (i64)pad - (i64)filt;
    if (stride < 1 || span < 0)
        return 0;
    i64 out = (span + stride - 1) / stride + 1;
    if (pad > 0 && (out - 1) * stride >= (i64)in + pad)
        out--;
    /* Without padding the rounded-up count can put the last window wholly
     * past the image (stride > filt): no input element, no pooling. */
    if ((out - 1) * stride - pad >= (i64)in)
        return 0;
    return (int)out;
}

/* Window of output index p along an axis: [lo, hi) inside the image and
 * the clipped padded area's extent. */
static void pool_window(int p, int stride, int pad, int filt, int in, i64 *lo, i64 *hi,
                        i64 *ext)
{
    i64 start = (i64)p * stride - pad;
    i64 end = start + filt;
    if (end > (i64)in + pad)
        end = (i64)in + pad;
    *ext = end - start;
    *lo = start < 0 ? 0 : start;
    *hi = end > in ? in : end;
}

void oracle_pool_fwd(int mode, int N, int C, int H, int W, int R, int S, int stride, int pad,
                     const double *x, double *y, double *ay, i64 *mask)
{
    int P = oracle_pool_out_size(H, R, stride, pad);
    int Q = oracle_pool_out_size(W, S, stride, pad);
    i64 nc;
#pragma omp parallel for schedule(static)
    for (nc = 0; nc < (i64)N * C; nc++) {
        const double *xp = x + nc * H * W;
        for (int p = 0; p < P; p++)
            for (int q = 0; q < Q; q++) {
                i64 h0, h1, eh, w0, w1, ew;
                pool_window(p, stride, pad, R, H, &h0, &h1, &eh);
                pool_window(q, stride, pad, S, W, &w0, &w1, &ew);
                i64 o = (nc * P + p) * Q + q;
                if (mode == 0) {
                    double best = -INFINITY;
                    i64 arg = -1;
                    for (i64 h = h0; h < h1; h++)
                        for (i64 w = w0; w < w1; w++)
                            if (xp[h * W + w] > best) {
                                best = xp[h * W + w];
                                arg = h * W + w;
                            }
                    y[o] = best;
                    if (ay)
                        ay[o] = fabs(best);
                    if (mask)
                        mask[o] = arg;
                } else {
                    double sum = 0.0, asum = 0.0;
                    for (i64 h = h0; h < h1; h++)
                        for (i64 w = w0; w < w1; w++) {
                            sum += xp[h * W + w];
                            asum += fabs(xp[h * W + w]);
                        }
                    double area = (double)(eh * ew);
                    y[o] = sum / area;
                    if (ay)
                        ay[o] = asum / area;
                }
            }
    }
}

void oracle_pool_bwd(int mode, int N, int C, int H, int W, int R, int S, int stride, int pad,
                     const double *dy, const i64 *mask, double *dx, double *adx)
{
    int P = oracle_pool_out_size(H, R, stride, pad);
    int Q = oracle_pool_out_size(W, S, stride, pad);
    i64 nc;
#pragma omp parallel for schedule(static)
    for (nc = 0; nc < (i64)N * C; nc++) {
        double *dxp = dx + nc * H * W;
        double *adxp = adx ? adx + nc * H * W : NULL;
        for (i64 i = 0; i < (i64)H * W; i++) {
            dxp[i] = 0.0;
            if (adxp)
                adxp[i] = 0.0;
        }
        for (int p = 0; p < P; p++)
            for (int q = 0; q < Q; q++) {
                i64 o = (nc * P + p) * Q + q;
                double g = dy[o];
                if (mode == 0) {
                    i64 arg = mask[o];
                    if (arg < 0 || arg >= (i64)H * W)
                        continue; /* the Python side rejects such masks first */
                    dxp[arg] += g;
                    if (adxp)
                        adxp[arg] += fabs(g);
                    continue;
                }
                i64 h0, h1, eh, w0, w1, ew;
                pool_window(p, stride, pad, R, H, &h0, &h1, &eh);
                pool_window(q, stride, pad, S, W, &w0, &w1, &ew);
                double share = g / (double)(eh * ew);
                for (i64 h = h0; h < h1; h++)
                    for (i64 w = w0; w < w1; w++) {
                        dxp[h * W + w] += share;
                        if (adxp)
                            adxp[h * W + w] += fabs(share);
                    }
            }
    }
}
