/*
 * oracle.c -- plain CPU reference of the CNN forward layers.
 *
 * TEST INFRASTRUCTURE: only the tests, the smoke check and the benchmark's
 * CPU-baseline leg load this library.  It shares no code with the GPU path.
 *
 * Every function is the direct definition of its layer, written as nested
 * loops in the order the definition reads, accumulating in double and
 * rounding each output once to float.  The paper lists the layer types
 * (Sec. 3.1) and verifies its library against Caffe on the last layer
 * (Sec. 4.1) but prints no formulas; where a convention is needed this file
 * follows Caffe's, which the paper's model-conversion path targets (Sec. 3.2).
 * OpenMP splits the outermost independent loops across threads; it changes
 * nothing in the order of any sum.
 */
#include "oracle.h"

#include <math.h>
#include <stddef.h>
#include <omp.h>

static int oracle_threads = 0; /* 0: OpenMP default */

void oracle_set_threads(int n) { oracle_threads = n > 0 ? n : 0; }

int oracle_get_threads(void) {
    return oracle_threads > 0 ? oracle_threads : omp_get_max_threads();
}

static float relu_f(float v) { return v > 0.0f ? v : 0.0f; }

/* Output size of a convolution: floor rule. */
int oracle_conv2d_out_shape(int H, int W, int R, int S, int sh, int sw,
                            int ph, int pw, int* P, int* Q) {
    if (H <= 0 || W <= 0 || R <= 0 || S <= 0 || sh <= 0 || sw <= 0 ||
        ph < 0 || pw < 0 || !P || !Q)
        return -1;
    if (H + 2 * ph < R || W + 2 * pw < S) return -1;
    *P = (H + 2 * ph - R) / sh + 1;
    *Q = (W + 2 * pw - S) / sw + 1;
    return 0;
}

/* One pooled extent: ceil (or floor) of the window count; in ceil mode a last
 * window that would start at or past the end of the image plus its padding
 * is dropped, so that every window holds at least one image element.  With
 * padding this is Caffe's rule; without padding it only matters when the
 * stride exceeds the window. */
static int pool_extent(int in, int k, int s, int pad, int ceil_mode) {
    int span = in + 2 * pad - k; /* >= 0 checked by the caller */
    int out = ceil_mode ? (span + s - 1) / s + 1 : span / s + 1;
    if (ceil_mode && (out - 1) * s >= in + pad) out -= 1;
    return out;
}

int oracle_pool_out_shape(int H, int W, int kh, int kw, int sh, int sw,
                          int ph, int pw, int ceil_mode, int* P, int* Q) {
    if (H <= 0 || W <= 0 || kh <= 0 || kw <= 0 || sh <= 0 || sw <= 0 ||
        ph < 0 || pw < 0 || ph >= kh || pw >= kw || !P || !Q)
        return -1;
    if (H + 2 * ph < kh || W + 2 * pw < kw) return -1;
    *P = pool_extent(H, kh, sh, ph, ceil_mode);
    *Q = pool_extent(W, kw, sw, pw, ceil_mode);
    return 0;
}

int oracle_conv2d_fwd(const float* x, int N, int C, int H, int W,
                      const float* w, int K, int R, int S, const float* bias,
                      int sh, int sw, int ph, int pw, int groups, int relu,
                      float* y) {
    int P, Q;
    if (!x || !w || !y || N < 0 || C <= 0 || K <= 0 || groups <= 0) return -1;
    if (C % groups != 0 || K % groups != 0) return -1;
    if (oracle_conv2d_out_shape(H, W, R, S, sh, sw, ph, pw, &P, &Q) != 0) return -1;
    const int Cg = C / groups; /* input channels per group */
    const int Kg = K / groups; /* output channels per group */

#pragma omp parallel for collapse(2) schedule(static) num_threads(oracle_get_threads())
    for (int n = 0; n < N; ++n) {
        for (int k = 0; k < K; ++k) {
            const int g = k / Kg;
            for (int p = 0; p < P; ++p) {
                for (int q = 0; q < Q; ++q) {
                    double acc = bias ? (double)bias[k] : 0.0;
                    for (int c = 0; c < Cg; ++c) {
                        const int ci = g * Cg + c;
                        for (int r = 0; r < R; ++r) {
                            const int h = p * sh - ph + r;
                            if (h < 0 || h >= H) continue; /* zero padding */
                            for (int s = 0; s < S; ++s) {
                                const int ww = q * sw - pw + s;
                                if (ww < 0 || ww >= W) continue;
                                const double xv =
                                    x[(((size_t)n * C + ci) * H + h) * W + ww];
                                const double wv =
                                    w[(((size_t)k * Cg + c) * R + r) * S + s];
                                acc += xv * wv;
                            }
                        }
                    }
                    float out = (float)acc;
                    if (relu) out = relu_f(out);
                    y[(((size_t)n * K + k) * P + p) * Q + q] = out;
                }
            }
        }
    }
    return 0;
}

int oracle_fc_fwd(const float* x, int N, int I, const float* w,
                  const float* bias, int O, int relu, float* y) {
    if (!x || !w || !y || N < 0 || I <= 0 || O <= 0) return -1;
#pragma omp parallel for collapse(2) schedule(static) num_threads(oracle_get_threads())
    for (int n = 0; n < N; ++n) {
        for (int o = 0; o < O; ++o) {
            double acc = bias ? (double)bias[o] : 0.0;
            for (int i = 0; i < I; ++i)
                acc += (double)x[(size_t)n * I + i] * (double)w[(size_t)o * I + i];
            float out = (float)acc;
            if (relu) out = relu_f(out);
            y[(size_t)n * O + o] = out;
        }
    }
    return 0;
}

int oracle_pool_fwd(const float* x, int N, int C, int H, int W, int mode,
                    int kh, int kw, int sh, int sw, int ph, int pw,
                    int ceil_mode, int relu, float* y, int32_t* idx) {
    int P, Q;
    if (!x || !y || N < 0 || C <= 0 || (mode != 0 && mode != 1)) return -1;
    if (oracle_pool_out_shape(H, W, kh, kw, sh, sw, ph, pw, ceil_mode, &P, &Q) != 0)
        return -1;

#pragma omp parallel for collapse(2) schedule(static) num_threads(oracle_get_threads())
    for (int n = 0; n < N; ++n) {
        for (int c = 0; c < C; ++c) {
            const float* plane = x + ((size_t)n * C + c) * H * W;
            for (int p = 0; p < P; ++p) {
                for (int q = 0; q < Q; ++q) {
                    const int hs = p * sh - ph, ws = q * sw - pw;
                    const size_t o = (((size_t)n * C + c) * P + p) * Q + q;
                    float out;
                    if (mode == 0) {
                        /* window clipped to the image; first maximum wins */
                        const int h0 = hs < 0 ? 0 : hs, w0 = ws < 0 ? 0 : ws;
                        const int h1 = hs + kh < H ? hs + kh : H;
                        const int w1 = ws + kw < W ? ws + kw : W;
                        float best = plane[(size_t)h0 * W + w0];
                        int best_i = h0 * W + w0;
                        for (int h = h0; h < h1; ++h)
                            for (int ww = w0; ww < w1; ++ww)
                                if (plane[(size_t)h * W + ww] > best) {
                                    best = plane[(size_t)h * W + ww];
                                    best_i = h * W + ww;
                                }
                        out = best;
                        if (idx) idx[o] = best_i;
                    } else {
                        /* divisor: window area within the padded extent */
                        const int h1p = hs + kh < H + ph ? hs + kh : H + ph;
                        const int w1p = ws + kw < W + pw ? ws + kw : W + pw;
                        const int count = (h1p - hs) * (w1p - ws);
                        const int h0 = hs < 0 ? 0 : hs, w0 = ws < 0 ? 0 : ws;
                        const int h1 = hs + kh < H ? hs + kh : H;
                        const int w1 = ws + kw < W ? ws + kw : W;
                        double sum = 0.0;
                        for (int h = h0; h < h1; ++h)
                            for (int ww = w0; ww < w1; ++ww)
                                sum += plane[(size_t)h * W + ww];
                        out = (float)(sum / count);
                    }
                    if (relu) out = relu_f(out);
                    y[o] = out;
                }
            }
        }
    }
    return 0;
}

int oracle_lrn_fwd(const float* x, int N, int C, int H, int W, int size,
                   float alpha, float beta, float k, float* y) {
    if (!x || !y || N < 0 || C <= 0 || H <= 0 || W <= 0) return -1;
    if (size <= 0 || size % 2 == 0) return -1;
    const int half = size / 2;
    const size_t HW = (size_t)H * W;

#pragma omp parallel for collapse(2) schedule(static) num_threads(oracle_get_threads())
    for (int n = 0; n < N; ++n) {
        for (int c = 0; c < C; ++c) {
            const int c0 = c - half < 0 ? 0 : c - half;
            const int c1 = c + half > C - 1 ? C - 1 : c + half;
            for (size_t hw = 0; hw < HW; ++hw) {
                double sq = 0.0;
                for (int cc = c0; cc <= c1; ++cc) {
                    const double v = x[((size_t)n * C + cc) * HW + hw];
                    sq += v * v;
                }
                const double scale = (double)k + (double)alpha / size * sq;
                const double v = x[((size_t)n * C + c) * HW + hw];
                y[((size_t)n * C + c) * HW + hw] = (float)(v * pow(scale, -(double)beta));
            }
        }
    }
    return 0;
}

int oracle_relu_fwd(const float* x, float* y, int64_t n) {
    if (!x || !y || n < 0) return -1;
    for (int64_t i = 0; i < n; ++i) y[i] = relu_f(x[i]);
    return 0;
}

/* Softmax across channels (Sec. 3.1 lists the layer; the definition is the
 * usual normalized exponential, over axis 1 as in Caffe): for every image n
 * and position i of the H*W plane,
 *   y[n,c,i] = exp(x[n,c,i]) / sum_{c'} exp(x[n,c',i]).
 * Both exponentials are taken of x - max_c' x[n,c',i], which leaves the
 * quotient unchanged and keeps exp from overflowing; everything in double,
 * rounded once. */
int oracle_softmax_fwd(const float* x, int N, int C, int HW, float* y) {
    if (N < 0 || C <= 0 || HW <= 0) return -1;
    if (N > 0 && (!x || !y)) return -1;
    int64_t cols = (int64_t)N * HW;
#pragma omp parallel for schedule(static)
    for (int64_t col = 0; col < cols; ++col) {
        const int64_t n = col / HW, i = col % HW;
        const int64_t cs = HW;  /* distance between channels */
        const float* xc = x + n * (int64_t)C * HW + i;
        float* yc = y + n * (int64_t)C * HW + i;
        double m = xc[0];
        for (int c = 1; c < C; ++c)
            if (xc[c * cs] > m) m = xc[c * cs];
        double sum = 0.0;
        for (int c = 0; c < C; ++c) sum += exp((double)xc[c * cs] - m);
        for (int c = 0; c < C; ++c) yc[c * cs] = (float)(exp((double)xc[c * cs] - m) / sum);
    }
    return 0;
}
