/*
 * caffe_ref.c -- plain CPU oracle for the Caffe convolution layer and the
 * pooling / local-response-normalisation glue that sits between conv layers.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke check and the CPU-baseline
 * leg of the benchmark may load this library.  It shares no code, header,
 * table or helper with the HIP library; nothing in the product path may call
 * it.
 *
 * What the paper fixes (Caffe, Jia et al. 2014, Sec. 3.2 "Layers"): a layer
 * maps input blobs to output blobs in its forward pass; its backward pass maps
 * the gradient w.r.t. the outputs to the gradients w.r.t. the parameters and
 * w.r.t. the inputs.  Blobs are 4-D arrays (Sec. 3.1), here N x C x H x W in
 * row-major order.  The paper gives no formula for convolution, so the
 * forward pass is the textbook strided, zero-padded, grouped 2-D
 * cross-correlation (no kernel flip), and the backward pass is its exact
 * derivative:
 *
 *   Ho = floor((H + 2 ph - kh) / sh) + 1,  Wo likewise,  Cg = C/G, Kg = K/G
 *   group of output channel k:  t = floor(k / Kg)
 *   Z[n,k,i,j] = b[k] + sum_{c<Cg,u<kh,v<kw} W[k,c,u,v] X[n, t Cg + c, i sh - ph + u, j sw - pw + v]
 *                (X read as 0 outside the image)
 *   Y = relu ? max(Z, 0) : Z
 *   D = relu ? G * [Y > 0] : G              (G = gradient w.r.t. Y)
 *   db[k]      = sum_{n,i,j} D[n,k,i,j]
 *   dW[k,c,u,v] = sum_{n,i,j} D[n,k,i,j] X[n, t Cg + c, i sh - ph + u, j sw - pw + v]
 *   dX[n, t Cg + c, i sh - ph + u, j sw - pw + v] += W[k,c,u,v] D[n,k,i,j]   (in-range positions)
 *
 * Weights are K x Cg x kh x kw (output channel major).  Every value is
 * double and every sum is accumulated in double in the plain loop order
 * written below.  Loops over independent outputs are spread over OpenMP
 * threads; no sum is ever split across threads, so results do not depend on
 * the thread count.
 *
 * Return value: 0 on success, -1 on an invalid shape (nothing is written).
 */
#include <math.h>
#include <stddef.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static long conv_out(long in, long k, long s, long p)
{
    return (in + 2 * p - k) / s + 1;
}

static int conv_shape_ok(int N, int C, int H, int W, int K, int kh, int kw, int sh, int sw,
                         int ph, int pw, int group)
{
    if (N < 0 || C < 1 || H < 1 || W < 1 || K < 1 || kh < 1 || kw < 1 || sh < 1 || sw < 1)
        return 0;
    if (ph < 0 || pw < 0 || group < 1 || C % group || K % group)
        return 0;
    if (H + 2 * ph < kh || W + 2 * pw < kw)
        return 0;
    return 1;
}

int caffe_ref_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int caffe_ref_conv_out_shape(int H, int W, int kh, int kw, int sh, int sw, int ph, int pw,
                             int* Ho, int* Wo)
{
    if (H < 1 || W < 1 || kh < 1 || kw < 1 || sh < 1 || sw < 1 || ph < 0 || pw < 0)
        return -1;
    if (H + 2 * ph < kh || W + 2 * pw < kw)
        return -1;
    *Ho = (int)conv_out(H, kh, sh, ph);
    *Wo = (int)conv_out(W, kw, sw, pw);
    return 0;
}

/* Forward pass of the convolution layer (Sec. 3.2: inputs -> outputs). */
int caffe_ref_conv_forward(int N, int C, int H, int W, int K, int kh, int kw, int sh, int sw,
                           int ph, int pw, int group, int relu,
                           const double* x, const double* w, const double* b, double* y)
{
    if (!conv_shape_ok(N, C, H, W, K, kh, kw, sh, sw, ph, pw, group))
        return -1;
    const long Ho = conv_out(H, kh, sh, ph), Wo = conv_out(W, kw, sw, pw);
    const long Cg = C / group, Kg = K / group;

#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (long n = 0; n < N; ++n) {
        for (long k = 0; k < K; ++k) {
            const long t = k / Kg;
            for (long i = 0; i < Ho; ++i) {
                for (long j = 0; j < Wo; ++j) {
                    double z = b ? b[k] : 0.0;
                    for (long c = 0; c < Cg; ++c) {
                        for (long u = 0; u < kh; ++u) {
                            const long ih = i * sh - ph + u;
                            if (ih < 0 || ih >= H)
                                continue;
                            for (long v = 0; v < kw; ++v) {
                                const long iw = j * sw - pw + v;
                                if (iw < 0 || iw >= W)
                                    continue;
                                z += w[((k * Cg + c) * kh + u) * kw + v] *
                                     x[((n * C + t * Cg + c) * H + ih) * W + iw];
                            }
                        }
                    }
                    if (relu && !(z > 0.0))
                        z = 0.0;
                    y[((n * K + k) * Ho + i) * Wo + j] = z;
                }
            }
        }
    }
    return 0;
}

/* Gradient w.r.t. the conv output after the (optional) ReLU: D = G [Y > 0]. */
static double masked_diff(const double* top, const double* top_diff, long idx, int relu)
{
    if (relu && !(top[idx] > 0.0))
        return 0.0;
    return top_diff[idx];
}

/*
 * Backward pass of the convolution layer (Sec. 3.2: output gradient ->
 * parameter gradients and input gradient).  Any of dx, dw, db may be NULL to
 * skip that gradient.  `top` (the forward output Y) is read only when relu is
 * set.  dx, dw and db are overwritten.
 */
int caffe_ref_conv_backward(int N, int C, int H, int W, int K, int kh, int kw, int sh, int sw,
                            int ph, int pw, int group, int relu,
                            const double* x, const double* w, const double* top,
                            const double* top_diff, double* dx, double* dw, double* db)
{
    if (!conv_shape_ok(N, C, H, W, K, kh, kw, sh, sw, ph, pw, group))
        return -1;
    if (relu && !top)
        return -1;
    const long Ho = conv_out(H, kh, sh, ph), Wo = conv_out(W, kw, sw, pw);
    const long Cg = C / group, Kg = K / group;

    if (db) {
#pragma omp parallel for schedule(static)
        for (long k = 0; k < K; ++k) {
            double s = 0.0;
            for (long n = 0; n < N; ++n)
                for (long i = 0; i < Ho; ++i)
                    for (long j = 0; j < Wo; ++j)
                        s += masked_diff(top, top_diff, ((n * K + k) * Ho + i) * Wo + j, relu);
            db[k] = s;
        }
    }

    if (dw) {
#pragma omp parallel for schedule(dynamic, 1)
        for (long k = 0; k < K; ++k) {
            const long t = k / Kg;
            double* dwk = dw + k * Cg * kh * kw;
            for (long r = 0; r < Cg * kh * kw; ++r)
                dwk[r] = 0.0;
            for (long n = 0; n < N; ++n) {
                for (long i = 0; i < Ho; ++i) {
                    for (long j = 0; j < Wo; ++j) {
                        const double d =
                            masked_diff(top, top_diff, ((n * K + k) * Ho + i) * Wo + j, relu);
                        for (long c = 0; c < Cg; ++c) {
                            for (long u = 0; u < kh; ++u) {
                                const long ih = i * sh - ph + u;
                                if (ih < 0 || ih >= H)
                                    continue;
                                for (long v = 0; v < kw; ++v) {
                                    const long iw = j * sw - pw + v;
                                    if (iw < 0 || iw >= W)
                                        continue;
                                    dwk[(c * kh + u) * kw + v] +=
                                        d * x[((n * C + t * Cg + c) * H + ih) * W + iw];
                                }
                            }
                        }
                    }
                }
            }
        }
    }

    if (dx) {
        /* Scatter form: each (image, group) pair owns a disjoint slice of dX. */
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
        for (long n = 0; n < N; ++n) {
            for (long t = 0; t < group; ++t) {
                double* dxs = dx + (n * C + t * Cg) * H * W;
                for (long e = 0; e < Cg * H * W; ++e)
                    dxs[e] = 0.0;
                for (long k = t * Kg; k < (t + 1) * Kg; ++k) {
                    for (long i = 0; i < Ho; ++i) {
                        for (long j = 0; j < Wo; ++j) {
                            const double d =
                                masked_diff(top, top_diff, ((n * K + k) * Ho + i) * Wo + j, relu);
                            for (long c = 0; c < Cg; ++c) {
                                for (long u = 0; u < kh; ++u) {
                                    const long ih = i * sh - ph + u;
                                    if (ih < 0 || ih >= H)
                                        continue;
                                    for (long v = 0; v < kw; ++v) {
                                        const long iw = j * sw - pw + v;
                                        if (iw < 0 || iw >= W)
                                            continue;
                                        dxs[(c * H + ih) * W + iw] +=
                                            w[((k * Cg + c) * kh + u) * kw + v] * d;
                                    }
                                }
                            }
                        }
                    }
                }
            }
        }
    }
    return 0;
}

/*
 * Max pooling (listed among Caffe's layer types in Sec. 3.2; used by the
 * LeNet example of Fig. 1).  Window rows i*s - p .. i*s - p + k - 1, clipped
 * to the image; output size floor((H + 2p - k)/s) + 1.  Ties go to the first
 * maximum in row-major window order (strict '>').  The backward pass routes
 * each output gradient to the input position that produced the maximum.
 */
static long pool_argmax(const double* plane, long H, long W, long i, long j, int k, int s, int p)
{
    long h0 = i * s - p, w0 = j * s - p;
    long h1 = h0 + k, w1 = w0 + k;
    if (h0 < 0) h0 = 0;
    if (w0 < 0) w0 = 0;
    if (h1 > H) h1 = H;
    if (w1 > W) w1 = W;
    long best = -1;
    double bv = 0.0;
    for (long h = h0; h < h1; ++h)
        for (long ww = w0; ww < w1; ++ww)
            if (best < 0 || plane[h * W + ww] > bv) {
                bv = plane[h * W + ww];
                best = h * W + ww;
            }
    return best;
}

static int pool_shape_ok(int N, int C, int H, int W, int k, int s, int p)
{
    if (N < 0 || C < 1 || H < 1 || W < 1 || k < 1 || s < 1 || p < 0 || p >= k)
        return 0;
    return H + 2 * p >= k && W + 2 * p >= k;
}

int caffe_ref_maxpool_forward(int N, int C, int H, int W, int k, int s, int p,
                              const double* x, double* y)
{
    if (!pool_shape_ok(N, C, H, W, k, s, p))
        return -1;
    const long Ho = conv_out(H, k, s, p), Wo = conv_out(W, k, s, p);
#pragma omp parallel for schedule(static)
    for (long nc = 0; nc < (long)N * C; ++nc) {
        const double* plane = x + nc * H * W;
        for (long i = 0; i < Ho; ++i)
            for (long j = 0; j < Wo; ++j) {
                const long a = pool_argmax(plane, H, W, i, j, k, s, p);
                y[(nc * Ho + i) * Wo + j] = plane[a];
            }
    }
    return 0;
}

int caffe_ref_maxpool_backward(int N, int C, int H, int W, int k, int s, int p,
                               const double* x, const double* top_diff, double* dx)
{
    if (!pool_shape_ok(N, C, H, W, k, s, p))
        return -1;
    const long Ho = conv_out(H, k, s, p), Wo = conv_out(W, k, s, p);
#pragma omp parallel for schedule(static)
    for (long nc = 0; nc < (long)N * C; ++nc) {
        const double* plane = x + nc * H * W;
        double* dplane = dx + nc * H * W;
        for (long e = 0; e < (long)H * W; ++e)
            dplane[e] = 0.0;
        for (long i = 0; i < Ho; ++i)
            for (long j = 0; j < Wo; ++j) {
                const long a = pool_argmax(plane, H, W, i, j, k, s, p);
                dplane[a] += top_diff[(nc * Ho + i) * Wo + j];
            }
    }
    return 0;
}

/*
 * Local response normalisation across channels (Sec. 3.2 layer list).
 *   s_c = kk + (alpha / size) * sum_{c' in win(c)} a_{c'}^2
 *   b_c = a_c * s_c^(-beta)
 * win(c) = channels c - (size-1)/2 ... c - (size-1)/2 + size - 1, clipped to
 * [0, C); the divisor stays `size` at the edges.  The backward pass is the
 * exact derivative:
 *   da_c = g_c s_c^(-beta)
 *          - (2 alpha beta / size) a_c sum_{c' : c in win(c')} g_{c'} b_{c'} / s_{c'}
 */
static void lrn_window(long c, long C, int size, long* lo, long* hi)
{
    long a = c - (size - 1) / 2, b = a + size; /* [a, b) */
    *lo = a < 0 ? 0 : a;
    *hi = b > C ? C : b;
}

static double lrn_scale(const double* col, long C, long HW, long c, int size, double alpha,
                        double kk)
{
    long lo, hi;
    lrn_window(c, C, size, &lo, &hi);
    double sq = 0.0;
    for (long q = lo; q < hi; ++q)
        sq += col[q * HW] * col[q * HW];
    return kk + alpha / size * sq;
}

int caffe_ref_lrn_forward(int N, int C, int H, int W, int size, double alpha, double beta,
                          double kk, const double* x, double* y)
{
    if (N < 0 || C < 1 || H < 1 || W < 1 || size < 1)
        return -1;
    const long HW = (long)H * W;
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; ++n)
        for (long c = 0; c < C; ++c)
            for (long e = 0; e < HW; ++e) {
                const double* col = x + n * C * HW + e;
                const double s = lrn_scale(col, C, HW, c, size, alpha, kk);
                y[(n * C + c) * HW + e] = col[c * HW] * pow(s, -beta);
            }
    return 0;
}

int caffe_ref_lrn_backward(int N, int C, int H, int W, int size, double alpha, double beta,
                           double kk, const double* x, const double* top_diff, double* dx)
{
    if (N < 0 || C < 1 || H < 1 || W < 1 || size < 1)
        return -1;
    const long HW = (long)H * W;
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; ++n)
        for (long c = 0; c < C; ++c)
            for (long e = 0; e < HW; ++e) {
                const double* col = x + n * C * HW + e;
                const double* gcol = top_diff + n * C * HW + e;
                const double s_c = lrn_scale(col, C, HW, c, size, alpha, kk);
                double cross = 0.0;
                for (long q = c - size + 1; q < c + size; ++q) { /* every c' whose window holds c */
                    if (q < 0 || q >= C)
                        continue;
                    long lo, hi;
                    lrn_window(q, C, size, &lo, &hi);
                    if (c < lo || c >= hi)
                        continue;
                    const double s_q = lrn_scale(col, C, HW, q, size, alpha, kk);
                    const double b_q = col[q * HW] * pow(s_q, -beta);
                    cross += gcol[q * HW] * b_q / s_q;
                }
                dx[(n * C + c) * HW + e] =
                    gcol[c * HW] * pow(s_c, -beta) - 2.0 * alpha * beta / size * col[c * HW] * cross;
            }
    return 0;
}
