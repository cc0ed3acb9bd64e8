// Device side of the bias fills (FillJobs, common.h): job j sets
// y_j[n][o][i] = bias_j[o] (or 0) for i < inner, shared out over every
// thread of the launch.  Element indices are below 2^31 (every tensor is),
// so (n, o) comes from two multiply-high divisions rather than 64-bit ones.
#pragma once

#include "common.h"

namespace cnn {

template <int CAP>
__device__ inline void run_fills(const FillJobsOf<CAP>& f) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int j = 0; j < f.n; ++j) {
        const BiasFill& jb = f.job[j];
        const int64_t total = jb.total;
        if (!jb.bias) {
            for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride)
                jb.y[i] = 0.0f;
            continue;
        }
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
            const unsigned row = fdiv((unsigned)i, jb.f_inner);  // n * O + o
            jb.y[i] = jb.bias[row - fdiv(row, jb.f_o) * (unsigned)jb.O];
        }
    }
}

}  // namespace cnn
