// Device side of the bias fills (FillJobs, common.h): job j sets
// y_j[n][o][i] = bias_j[o] (or 0) for i < inner, shared out over every
// thread of the launch.
#pragma once

#include "common.h"

namespace cnn {

__device__ inline void run_fills(const FillJobs& f) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int j = 0; j < f.n; ++j) {
        const BiasFill& jb = f.job[j];
        const int64_t total = (int64_t)jb.N * jb.O * jb.inner;
        for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride)
            jb.y[i] = jb.bias ? jb.bias[(i / jb.inner) % jb.O] : 0.0f;
    }
}

}  // namespace cnn
