// Convolution configuration table, heuristic choice and launcher; the kernel
// template is in conv_igemm_kernel.h and its instantiations are spread over
// conv_cfg_*.hip so that they compile in parallel.
#include <algorithm>

#include "conv_igemm_kernel.h"

namespace cnn {
namespace conv {
namespace {

struct ConvConfig {
    const char* name;  // "TMxTNxBK"
    int tm, tn, bk, threads;
    LaunchFn launch;
};

#define CNN_CONV_ENTRY(I, WMW, WNW, FM, FN, BK)                                            \
    ConvConfig{#WMW "x" #WNW " waves, " #FM "x" #FN " blocks, BK " #BK, WMW * FM * 32, WNW * FN * 32, \
               BK, 64 * WMW * WNW, &launch_c##I},

const ConvConfig kConfigs[] = {CNN_CONV_CONFIGS(CNN_CONV_ENTRY)};
constexpr int kNumConfigs = sizeof(kConfigs) / sizeof(kConfigs[0]);

// Heuristic choice when no tuned entry exists: the output-channel tile follows
// the group's channel count; a narrower pixel tile when the grid would leave
// most compute units idle.
int heuristic_config(const ConvParams& p, int G) {
    const int mt128 = ceil_div(p.M, 128);
    if (p.Kg <= 32) return 8;
    if (p.Kg <= 64) return mt128 * G >= 512 ? 4 : 9;
    if (p.Kg <= 96) return 6;
    const int blocks = mt128 * ceil_div(p.Kg, 128) * G;
    return blocks >= 512 ? 0 : 2;
}

}  // namespace
}  // namespace conv

using conv::ConvParams;
using conv::kConfigs;
using conv::kNumConfigs;
using conv::heuristic_config;

int conv2d_num_configs() { return kNumConfigs; }

const char* conv2d_config_name(int i) { return (i >= 0 && i < kNumConfigs) ? kConfigs[i].name : nullptr; }

int launch_conv2d(const ConvShape& s, const float* x, const float* w, const float* bias, int relu,
                  float* y, hipStream_t st, int cfg) {
    ConvParams prm;
    prm.w = w;
    prm.bias = bias;
    prm.C = s.C; prm.H = s.H; prm.W = s.W; prm.K = s.K; prm.R = s.R; prm.S = s.S;
    prm.P = s.P; prm.Q = s.Q;
    prm.sh = s.sh; prm.sw = s.sw; prm.ph = s.ph; prm.pw = s.pw;
    prm.Cg = s.C / s.G;
    prm.Kg = s.K / s.G;
    prm.RS = s.R * s.S;
    prm.Kr = prm.Cg * prm.RS;
    prm.HW = s.H * s.W;
    prm.PQ = s.P * s.Q;
    prm.relu = relu;
    if (s.N == 0) return CNN_OK;
    const bool vec_w = (prm.Kr % 4 == 0) && ((reinterpret_cast<uintptr_t>(w) & 15) == 0);
    const int64_t wbytes = (int64_t)s.K * prm.Kr * 4;
    if (wbytes >= ((int64_t)1 << 31)) return fail(CNN_ERR_UNSUPPORTED, "conv: weights exceed 2 GiB");
    prm.wbytes = (int)wbytes;

    // The gather addresses x through a buffer resource with 31-bit offsets:
    // launch fewer than 2^29 input elements at a time (whole images).
    const int64_t img = (int64_t)s.C * prm.HW;
    const int per_launch = (int)std::min<int64_t>(s.N, (((int64_t)1 << 29) - 1) / img);
    if (per_launch < 1) return fail(CNN_ERR_UNSUPPORTED, "conv: one image exceeds 2^29 elements");
    if (cfg < 0) {
        prm.M = per_launch * prm.PQ;
        cfg = heuristic_config(prm, s.G);
    }
    if (cfg >= kNumConfigs) return fail(CNN_ERR_UNSUPPORTED, "conv: no configuration %d", cfg);
    for (int n0 = 0; n0 < s.N; n0 += per_launch) {
        const int nb = std::min(per_launch, s.N - n0);
        prm.x = x + (size_t)n0 * img;
        prm.y = y + (size_t)n0 * s.K * prm.PQ;
        prm.M = nb * prm.PQ;
        prm.xbytes = (int)(nb * img * 4);
        const int rc = kConfigs[cfg].launch(prm, s.G, vec_w, st);
        if (rc != CNN_OK) return rc;
    }
    return CNN_OK;
}

}  // namespace cnn
