/* The C ABI used from C alone (no Python, no torch): the CIFAR-10 quick
 * network (the paper's layer-setup table, Sec. 4) is described with
 * cnn_layer_desc, run on the GPU with cnn_net_fwd on buffers from the HIP
 * runtime, and compared with the oracle's layers chained on the host.
 *
 * Inputs: a counter-based generator (SplitMix64, Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014) mapped to
 * [0, 1) for the image and to roughly N(0, std) (sum of four uniforms,
 * centred and scaled) for weights and biases.  The same bytes go to both
 * sides.
 *
 * Pass: max |gpu - oracle| <= 1e-4 * sqrt(64) and relative L2 <= 1e-4 on the
 * 32 x 10 logits (the FC criterion of the last layer, Kred = 64).  A second
 * pass through cnn_net_fwd_kernel_timed, with one pair of HIP events per
 * layer, must give the same logits (within that tolerance: split reductions
 * may add in another order) and a non-negative kernel time for every layer.
 * Exit status 0 on pass, 1 on a mismatch, 2 on an API or runtime error. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "cnn.h"
#include "oracle.h"

static uint64_t g_state;
static uint64_t splitmix64(void) {
    uint64_t z = (g_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}
static float uniform01(void) { return (float)(splitmix64() >> 40) / (float)(1u << 24); }
static float normalish(float std) {  /* variance of a sum of 4 uniforms: 4/12 */
    float s = uniform01() + uniform01() + uniform01() + uniform01() - 2.0f;
    return s * std * 1.7320508f;
}
static float* host_fill(size_t n, int normal, float std) {
    float* a = (float*)malloc(n * sizeof(float));
    for (size_t i = 0; i < n; ++i) a[i] = normal ? normalish(std) : uniform01();
    return a;
}

#define HIP_OK(call)                                                        \
    do {                                                                    \
        if ((call) != hipSuccess) {                                         \
            fprintf(stderr, "HIP error at %s:%d\n", __FILE__, __LINE__);     \
            return 2;                                                       \
        }                                                                   \
    } while (0)
#define CNN_OK_(call)                                                       \
    do {                                                                    \
        if ((call) != CNN_OK) {                                             \
            fprintf(stderr, "cnn error: %s\n", cnn_last_error());           \
            return 2;                                                       \
        }                                                                   \
    } while (0)

static float* to_device(const float* h, size_t n) {
    float* d = NULL;
    if (hipMalloc((void**)&d, n * sizeof(float)) != hipSuccess) return NULL;
    if (hipMemcpy(d, h, n * sizeof(float), hipMemcpyHostToDevice) != hipSuccess) return NULL;
    return d;
}

int main(void) {
    enum { N = 32, NL = 8 };
    g_state = 20151123ull;
    /* conv 32 5x5 p2 | maxpool 3/2 + ReLU | conv 32 5x5 p2 + ReLU | avgpool 3/2 |
     * conv 64 5x5 p2 + ReLU | avgpool 3/2 | FC 1024 -> 64 | FC 64 -> 10 */
    const int conv_c[3] = {3, 32, 32}, conv_k[3] = {32, 32, 64}, conv_relu[3] = {0, 1, 1};
    const int fc_i[2] = {1024, 64}, fc_o[2] = {64, 10};
    float* w_h[5]; float* b_h[5]; float* w_d[5]; float* b_d[5];
    for (int i = 0; i < 3; ++i) {
        w_h[i] = host_fill((size_t)conv_k[i] * conv_c[i] * 25, 1, 0.05f);
        b_h[i] = host_fill((size_t)conv_k[i], 1, 0.01f);
    }
    for (int i = 0; i < 2; ++i) {
        w_h[3 + i] = host_fill((size_t)fc_o[i] * fc_i[i], 1, 0.05f);
        b_h[3 + i] = host_fill((size_t)fc_o[i], 1, 0.01f);
    }
    float* x_h = host_fill((size_t)N * 3 * 32 * 32, 0, 0.0f);
    for (int i = 0; i < 5; ++i) {
        const size_t nw = i < 3 ? (size_t)conv_k[i] * conv_c[i] * 25 : (size_t)fc_o[i - 3] * fc_i[i - 3];
        const size_t nb = i < 3 ? (size_t)conv_k[i] : (size_t)fc_o[i - 3];
        w_d[i] = to_device(w_h[i], nw);
        b_d[i] = to_device(b_h[i], nb);
        if (!w_d[i] || !b_d[i]) return 2;
    }

    cnn_layer_desc L[NL];
    memset(L, 0, sizeof(L));
    const int order[NL] = {CNN_LAYER_CONV, CNN_LAYER_POOL, CNN_LAYER_CONV, CNN_LAYER_POOL,
                           CNN_LAYER_CONV, CNN_LAYER_POOL, CNN_LAYER_FC, CNN_LAYER_FC};
    int ci = 0, fi = 0, pi = 0;
    for (int i = 0; i < NL; ++i) {
        L[i].type = order[i];
        if (order[i] == CNN_LAYER_CONV) {
            L[i].out_channels = conv_k[ci]; L[i].in_channels = conv_c[ci];
            L[i].kernel_h = L[i].kernel_w = 5; L[i].stride_h = L[i].stride_w = 1;
            L[i].pad_h = L[i].pad_w = 2; L[i].groups = 1; L[i].fuse_relu = conv_relu[ci];
            L[i].weight = w_d[ci]; L[i].bias = b_d[ci];
            ++ci;
        } else if (order[i] == CNN_LAYER_POOL) {
            L[i].pool_mode = pi == 0 ? CNN_POOL_MAX : CNN_POOL_AVG;
            L[i].kernel_h = L[i].kernel_w = 3; L[i].stride_h = L[i].stride_w = 2;
            L[i].ceil_mode = 1; L[i].fuse_relu = pi == 0;  /* Pooling+ReLU */
            ++pi;
        } else {
            L[i].out_channels = fc_o[fi]; L[i].in_features = fc_i[fi];
            L[i].weight = w_d[3 + fi]; L[i].bias = b_d[3 + fi];
            ++fi;
        }
    }

    int oc, oh, ow;
    CNN_OK_(cnn_net_out_shape(L, NL, N, 3, 32, 32, &oc, &oh, &ow));
    if (oc != 10 || oh != 1 || ow != 1) {
        fprintf(stderr, "unexpected output shape %dx%dx%d\n", oc, oh, ow);
        return 1;
    }
    const size_t ws_bytes = cnn_net_workspace_bytes(L, NL, N, 3, 32, 32);
    if (ws_bytes == 0) return 2;
    void* ws = NULL;
    float* y_d = NULL;
    float* x_d = to_device(x_h, (size_t)N * 3 * 32 * 32);
    if (!x_d) return 2;
    HIP_OK(hipMalloc(&ws, ws_bytes));
    HIP_OK(hipMalloc((void**)&y_d, (size_t)N * 10 * sizeof(float)));
    hipStream_t st;
    HIP_OK(hipStreamCreate(&st));
    CNN_OK_(cnn_net_fwd(L, NL, x_d, N, 3, 32, 32, y_d, ws, ws_bytes, (cnn_stream_t)st));
    HIP_OK(hipStreamSynchronize(st));
    float y_g[N * 10];
    HIP_OK(hipMemcpy(y_g, y_d, sizeof(y_g), hipMemcpyDeviceToHost));

    /* the same pass again, each layer timed by its kernels' own timestamps */
    hipEvent_t ev_start[NL], ev_stop[NL];
    void* starts[NL];
    void* stops[NL];
    for (int i = 0; i < NL; ++i) {
        HIP_OK(hipEventCreate(&ev_start[i]));
        HIP_OK(hipEventCreate(&ev_stop[i]));
        starts[i] = ev_start[i];
        stops[i] = ev_stop[i];
    }
    float* y2_d = NULL;
    HIP_OK(hipMalloc((void**)&y2_d, (size_t)N * 10 * sizeof(float)));
    CNN_OK_(cnn_net_fwd_kernel_timed(L, NL, x_d, N, 3, 32, 32, y2_d, ws, ws_bytes, starts, stops,
                                     (cnn_stream_t)st));
    HIP_OK(hipStreamSynchronize(st));
    float y_t[N * 10];
    HIP_OK(hipMemcpy(y_t, y2_d, sizeof(y_t), hipMemcpyDeviceToHost));
    float span_ms[NL];
    for (int i = 0; i < NL; ++i) {
        HIP_OK(hipEventElapsedTime(&span_ms[i], ev_start[i], ev_stop[i]));
        if (!(span_ms[i] >= 0.0f)) {
            fprintf(stderr, "layer %d: kernel interval %g ms\n", i, span_ms[i]);
            return 1;
        }
    }
    double timed_diff = 0.0;
    for (int i = 0; i < N * 10; ++i) timed_diff = fmax(timed_diff, fabs((double)y_t[i] - (double)y_g[i]));

    /* the oracle, layer by layer, ReLU as separate steps */
    float* a = (float*)malloc((size_t)N * 32 * 32 * 32 * sizeof(float));
    float* b = (float*)malloc((size_t)N * 32 * 32 * 32 * sizeof(float));
    int C = 3, H = 32, W = 32, P, Q;
    memcpy(a, x_h, (size_t)N * 3 * 32 * 32 * sizeof(float));
    ci = fi = pi = 0;
    for (int i = 0; i < NL; ++i) {
        if (order[i] == CNN_LAYER_CONV) {
            if (oracle_conv2d_out_shape(H, W, 5, 5, 1, 1, 2, 2, &P, &Q)) return 2;
            if (oracle_conv2d_fwd(a, N, C, H, W, w_h[ci], conv_k[ci], 5, 5, b_h[ci], 1, 1, 2, 2, 1, 0, b)) return 2;
            C = conv_k[ci]; H = P; W = Q;
            if (conv_relu[ci]) oracle_relu_fwd(b, b, (int64_t)N * C * H * W);
            ++ci;
        } else if (order[i] == CNN_LAYER_POOL) {
            if (oracle_pool_out_shape(H, W, 3, 3, 2, 2, 0, 0, 1, &P, &Q)) return 2;
            if (oracle_pool_fwd(a, N, C, H, W, pi == 0 ? 0 : 1, 3, 3, 2, 2, 0, 0, 1, 0, b, NULL)) return 2;
            H = P; W = Q;
            if (pi == 0) oracle_relu_fwd(b, b, (int64_t)N * C * H * W);
            ++pi;
        } else {
            if (oracle_fc_fwd(a, N, C * H * W, w_h[3 + fi], b_h[3 + fi], fc_o[fi], 0, b)) return 2;
            C = fc_o[fi]; H = W = 1;
            ++fi;
        }
        float* t = a; a = b; b = t;
    }

    double max_err = 0.0, num = 0.0, den = 0.0;
    for (int i = 0; i < N * 10; ++i) {
        const double d = (double)y_g[i] - (double)a[i];
        if (!isfinite(y_g[i])) max_err = INFINITY;
        if (fabs(d) > max_err) max_err = fabs(d);
        num += d * d;
        den += (double)a[i] * a[i];
    }
    const double rel = den > 0 ? sqrt(num / den) : 0.0;
    const double tol = 1e-4 * sqrt(64.0);
    printf("cifar_quick_c: %s, N=%d, max abs err %.3e (tol %.3e), rel L2 %.3e; kernel-timed pass differs by "
           "%.3e, layer kernel times (us):", cnn_version(), N, max_err, tol, rel, timed_diff);
    for (int i = 0; i < NL; ++i) printf(" %.1f", 1000.0 * span_ms[i]);
    printf("\n");
    for (int i = 0; i < NL; ++i) { hipEventDestroy(ev_start[i]); hipEventDestroy(ev_stop[i]); }
    hipStreamDestroy(st);
    hipFree(ws); hipFree(y_d); hipFree(y2_d); hipFree(x_d);
    for (int i = 0; i < 5; ++i) { hipFree(w_d[i]); hipFree(b_d[i]); free(w_h[i]); free(b_h[i]); }
    free(x_h); free(a); free(b);
    return (max_err <= tol && rel <= 1e-4 && timed_diff <= tol) ? 0 : 1;
}
