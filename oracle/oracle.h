/*
 * oracle.h -- plain CPU reference of the CNN forward layers.
 *
 * TEST INFRASTRUCTURE.  This library exists to check the GPU path.  Only the
 * tests, the smoke check and the benchmark's CPU-baseline leg may load it; the
 * product path never calls it and shares no code with it.
 *
 * The paper names the layer types (Sec. 3.1: convolution, max/mean pooling,
 * fully connected, ReLU, local response normalization, softmax) and checks its
 * implementation by running the same input through it and through Caffe and
 * comparing the last layer (Sec. 4.1).  It gives no formulas; every formula
 * here is the plain textbook definition, with Caffe's conventions where a
 * convention has to be picked.  Each function states its definition.
 *
 * Arithmetic: every sum is accumulated in double precision and every layer
 * output is rounded once to float, matching the paper's 32-bit storage
 * (Sec. 4.2).  Layout: NCHW, row-major, contiguous; host pointers.
 *
 * Return value: 0 on success, -1 for an invalid argument (nothing written).
 */
#ifndef CNN_ORACLE_H
#define CNN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Conv output size, floor rule: P = (H + 2*ph - R) / sh + 1. */
int oracle_conv2d_out_shape(int H, int W, int R, int S, int sh, int sw,
                            int ph, int pw, int* P, int* Q);

/* Pool output size.  ceil_mode=1: P = ceil((H + 2*ph - kh) / sh) + 1, and the
 * last window is dropped when it would start at or past H + ph (inside the
 * bottom/right padding); ceil_mode=0: floor instead of ceil.  Requires
 * ph < kh, so that every window overlaps the image. */
int oracle_pool_out_shape(int H, int W, int kh, int kw, int sh, int sw,
                          int ph, int pw, int ceil_mode, int* P, int* Q);

/* Grouped 2-D cross-correlation with stride, zero padding and bias:
 *   y[n,k,p,q] = b[k] + sum_{c<C/G, r<R, s<S}
 *                x[n, g*C/G + c, p*sh - ph + r, q*sw - pw + s] * w[k,c,r,s]
 * with g = k / (K/G) and x = 0 outside the image.  w is [K][C/G][R][S],
 * bias [K] or NULL, y [N][K][P][Q].  relu=1 applies y = max(y, 0) after
 * rounding. */
int oracle_conv2d_fwd(const float* x, int N, int C, int H, int W,
                      const float* w, int K, int R, int S, const float* bias,
                      int sh, int sw, int ph, int pw, int groups, int relu,
                      float* y);

/* Fully connected: y[n,o] = b[o] + sum_i x[n,i] * w[o,i].  x is [N][I] (a
 * flattened NCHW tensor: i = c*H*W + h*W + w), w [O][I], bias [O] or NULL. */
int oracle_fc_fwd(const float* x, int N, int I, const float* w,
                  const float* bias, int O, int relu, float* y);

/* Pooling over windows rows [p*sh - ph, p*sh - ph + kh) clipped to [0, H)
 * (columns alike).  mode 0 = max: value is the window maximum, idx (optional,
 * int32 [N][C][P][Q]) is h*W + w of the first maximum in row-major scan order.
 * mode 1 = average: sum of the clipped window divided by the window area
 * clipped to the padded extent [-ph, H + ph) x [-pw, W + pw).  relu=1 applies
 * max(y, 0) after pooling; the index is the pre-ReLU argmax. */
int oracle_pool_fwd(const float* x, int N, int C, int H, int W, int mode,
                    int kh, int kw, int sh, int sw, int ph, int pw,
                    int ceil_mode, int relu, float* y, int32_t* idx);

/* Local response normalization across channels, odd size n:
 *   y[n,c,h,w] = x[n,c,h,w] * (k + alpha/size * sum_{c'} x[n,c',h,w]^2)^(-beta)
 * with c' over [c - size/2, c + size/2] clipped to [0, C). */
int oracle_lrn_fwd(const float* x, int N, int C, int H, int W, int size,
                   float alpha, float beta, float k, float* y);

/* y[i] = x[i] > 0 ? x[i] : +0.0f */
int oracle_relu_fwd(const float* x, float* y, int64_t n);

/* Softmax across channels of x viewed as [N][C][HW] (HW = H*W; 1 after a
 * fully connected layer):
 *   y[n,c,i] = exp(x[n,c,i] - m) / sum_{c'} exp(x[n,c',i] - m),
 *   m = max_{c'} x[n,c',i]. */
int oracle_softmax_fwd(const float* x, int N, int C, int HW, float* y);

/* OpenMP threads used by the loops above (default: all). */
void oracle_set_threads(int n);
int oracle_get_threads(void);

#ifdef __cplusplus
}
#endif
#endif
