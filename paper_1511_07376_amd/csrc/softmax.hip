// Softmax layer across channels, for x viewed as [N][C][HW]:
//     y[n,c,i] = exp(x[n,c,i] - m) / sum_c' exp(x[n,c',i] - m),  m = max_c' x[n,c',i]
// (subtracting the column maximum leaves the quotient unchanged and keeps the
// exponential finite).  A few kilobytes per image after the last fully
// connected layer, so the kernels aim at latency: one pass for the maximum,
// one for the sum, one to write, all over data that stays in cache.
#include "common.h"

#include <algorithm>
#include <cmath>

namespace cnn {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ inline float wave_max(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
    return v;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// HW == 1 (the output of a fully connected layer): one wavefront per row of C
// contiguous values, lanes on consecutive channels.  Each element is read and
// then written by the same lane, so y == x works.
__global__ void __launch_bounds__(kThreads) softmax_rows_f32(const float* x, float* y, int rows, int C) {
    const int row = blockIdx.x * kWaves + (int)(threadIdx.x >> 6);  // uniform per wave
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const float* xr = x + (size_t)row * C;
    float* yr = y + (size_t)row * C;
    // 64-bit channel counters: a row may hold up to 2^31-1 values
    float m = -INFINITY;
    for (int64_t c = lane; c < C; c += 64) m = fmaxf(m, xr[c]);
    m = wave_max(m);
    float s = 0.0f;
    for (int64_t c = lane; c < C; c += 64) s += expf(xr[c] - m);
    s = wave_sum(s);
    for (int64_t c = lane; c < C; c += 64) yr[c] = expf(xr[c] - m) / s;
}

// HW > 1: one thread per (n, i) column, lanes on consecutive positions i of
// the plane (coalesced), looping over the channels.
__global__ void __launch_bounds__(kThreads) softmax_cols_f32(const float* x, float* y, int N, int C, int HW) {
    const int64_t col = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (col >= (int64_t)N * HW) return;
    const int n = (int)(col / HW);
    const int i = (int)(col - (int64_t)n * HW);
    const float* xc = x + (size_t)n * C * HW + i;
    float* yc = y + (size_t)n * C * HW + i;
    float m = -INFINITY;
    for (int c = 0; c < C; ++c) m = fmaxf(m, xc[(size_t)c * HW]);
    float s = 0.0f;
    for (int c = 0; c < C; ++c) s += expf(xc[(size_t)c * HW] - m);
    for (int c = 0; c < C; ++c) yc[(size_t)c * HW] = expf(xc[(size_t)c * HW] - m) / s;
}

}  // namespace

int launch_softmax(const float* x, int N, int C, int HW, float* y, hipStream_t st) {
    if (N == 0) return CNN_OK;
    if (HW == 1) {
        enqueue(softmax_rows_f32, dim3(ceil_div(N, kWaves)), dim3(kThreads), 0, st, x, y, N, C);
    } else {
        const int64_t cols = (int64_t)N * HW;
        enqueue(softmax_cols_f32, dim3((unsigned)ceil_div64(cols, kThreads)), dim3(kThreads), 0, st,
                           x, y, N, C, HW);
    }
    return check_launch("softmax_f32");
}

}  // namespace cnn
