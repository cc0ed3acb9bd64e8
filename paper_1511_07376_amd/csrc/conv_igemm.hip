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

#define CNN_CONV_ENTRY(I, WMW, WNW, FM, FN, BK, KS, ST)                                        \
    ConvConfig{#WMW "x" #WNW " waves, " #FM "x" #FN " blocks, BK " #BK ", " #KS " slab groups",      \
               WMW * FM * 32, WNW * FN * 32, BK, 64 * WMW * WNW * KS, &launch_c##I},

const ConvConfig kConfigs[] = {CNN_CONV_CONFIGS(CNN_CONV_ENTRY)};
constexpr int kNumConfigs = sizeof(kConfigs) / sizeof(kConfigs[0]);

// Heuristic choice when no tuned entry exists, fitted by hand to measured
// times of every configuration on AlexNet's, LeNet's and CIFAR-10 quick's
// layers and the single-layer sweep shapes at batches 1 to 256 (`python
// bench.py --config-table` times them all: over those 46 shapes the
// heuristic's total came within 0.5% of always picking the fastest on the
// box it was fitted on, and 4.0-4.9% over on others).  t64: output tiles of a
// 64 x 64 tile; b128: of a 128 x 128 tile.
int heuristic_config(const ConvParams& p, int G) {
    const int64_t t64 = (int64_t)ceil_div(p.M, 64) * ceil_div(p.Kg, 64) * G;
    const int64_t b128 = (int64_t)ceil_div(p.M, 128) * ceil_div(p.Kg, 128) * G;
    if (p.Kg <= 32) return 8;                                         // 32 x 128
    if (std::max(p.sh, p.sw) >= 4 && p.Kg > 64) return t64 >= 4000 ? 6 : 8;  // strided stem
    if (t64 >= 4000 && p.Kg > 64) return 4;                          // 64 x 128
    if (p.Kg > 64 && p.Kg <= 128 && b128 >= 512) return 0;           // 128 x 128
    if (p.Kg >= 256 && t64 >= 300 && t64 < 1000) return 2;           // 128 x 64
    if (t64 < 1000) return 10;                                        // 64 x 64, BK 32
    return 9;                                                         // 64 x 64, BK 16
}

// Reduction chunks for a configuration: when its output tiles would give the
// 256 compute units fewer than 1.5 workgroups each, split the reduction so
// that about 1024 workgroups run, keeping at least 8 slabs per chunk.  (On
// AlexNet at batch 16 this made conv3-conv5 25-32% faster than splitting
// only below 128 tiles into 512 workgroups; batches 1, 64 and 256 measured
// the same.)
constexpr int kSplitBelowTiles = 384, kSplitTarget = 1024;
void choose_splits(ConvParams& p, const ConvConfig& c) {
    const int tiles = ceil_div(p.M, c.tn) * ceil_div(p.Kg, c.tm) * p.G;
    const int nslab = ceil_div(p.Kr, c.bk);
    int splits = 1;
    if (tiles <= kSplitBelowTiles) splits = std::max(1, std::min(ceil_div(kSplitTarget, tiles), nslab / 8));
    const int slabs_per_chunk = ceil_div(nslab, splits);
    p.kchunk = splits > 1 ? slabs_per_chunk * c.bk : p.Kr;
    p.splits = splits > 1 ? ceil_div(p.Kr, p.kchunk) : 1;
}

}  // namespace
}  // namespace conv

using conv::ConvParams;
using conv::kConfigs;
using conv::kNumConfigs;
using conv::heuristic_config;
using conv::choose_splits;

int conv2d_num_configs() { return kNumConfigs; }

const char* conv2d_config_name(int i) { return (i >= 0 && i < kNumConfigs) ? kConfigs[i].name : nullptr; }

namespace {

// Parameters, configuration and reduction split of a convolution; per_launch:
// images per launch (the gather's 31-bit offsets cover fewer than 2^29 input
// elements).  cfg < 0 on entry: the heuristic's choice.
int conv_prepare(const ConvShape& s, int* cfg, ConvParams* out, int* per_launch) {
    ConvParams& prm = *out;
    prm.C = s.C; prm.H = s.H; prm.W = s.W; prm.K = s.K; prm.R = s.R; prm.S = s.S;
    prm.P = s.P; prm.Q = s.Q;
    prm.sh = s.sh; prm.sw = s.sw; prm.ph = s.ph; prm.pw = s.pw;
    prm.Cg = s.C / s.G;
    prm.Kg = s.K / s.G;
    prm.RS = s.R * s.S;
    prm.Kr = prm.Cg * prm.RS;
    prm.HW = s.H * s.W;
    prm.PQ = s.P * s.Q;
    prm.f_rs = make_fastdiv(prm.RS);
    prm.f_s = make_fastdiv(s.S);
    prm.f_pq = make_fastdiv(prm.PQ);
    prm.f_q = make_fastdiv(s.Q);
    prm.G = s.G;
    prm.splits = 1;
    prm.kchunk = prm.Kr;
    prm.relu_x = 0;
    const int64_t wbytes = (int64_t)s.K * prm.Kr * 4;
    if (wbytes >= ((int64_t)1 << 31)) return fail(CNN_ERR_UNSUPPORTED, "conv: weights exceed 2 GiB");
    prm.wbytes = (int)wbytes;
    const int64_t img = (int64_t)s.C * prm.HW;
    *per_launch = (int)std::min<int64_t>(std::max(s.N, 1), (((int64_t)1 << 29) - 1) / img);
    if (*per_launch < 1) return fail(CNN_ERR_UNSUPPORTED, "conv: one image exceeds 2^29 elements");
    prm.M = *per_launch * prm.PQ;
    if (*cfg < 0) *cfg = heuristic_config(prm, s.G);
    if (*cfg >= kNumConfigs) return fail(CNN_ERR_UNSUPPORTED, "conv: no configuration %d", *cfg);
    // One split decision for every launch of the call (the last one may hold
    // fewer images: splitting it the same way is still correct).
    choose_splits(prm, kConfigs[*cfg]);
    return CNN_OK;
}

}  // namespace

int conv2d_heuristic_config(const ConvShape& s) {
    ConvParams prm;
    int per_launch, cfg = -1;
    return conv_prepare(s, &cfg, &prm, &per_launch) == CNN_OK ? cfg : -1;
}

int conv2d_splits(const ConvShape& s, int cfg) {
    ConvParams prm;
    int per_launch;
    if (conv_prepare(s, &cfg, &prm, &per_launch) != CNN_OK) return 1;
    return prm.splits;
}

int launch_conv2d(const ConvShape& s, const float* x, const float* w, const float* bias, int relu,
                  float* y, hipStream_t st, int cfg, const ConvOpts* opt) {
    if (opt && opt->relu_left) *opt->relu_left = false;
    if (s.N == 0) return CNN_OK;
    ConvParams prm;
    int per_launch;
    int rc = conv_prepare(s, &cfg, &prm, &per_launch);
    if (rc != CNN_OK) return rc;
    prm.w = w;
    prm.bias = bias;
    prm.relu = relu;
    prm.relu_x = opt && opt->relu_in;
    const bool vec_w = (prm.Kr % 4 == 0) && ((reinterpret_cast<uintptr_t>(w) & 15) == 0);
    const int64_t img = (int64_t)s.C * prm.HW;
    const int64_t total = (int64_t)s.N * s.K * prm.PQ;
    if (prm.splits > 1 && !(opt && opt->prefilled)) {  // y[n][k][pq] = bias[k]: the sums' start
        const BiasFill fill = make_bias_fill(y, bias, s.N, s.K, prm.PQ);
        rc = launch_bias_fills(&fill, 1, st);
        if (rc != CNN_OK) return rc;
    }
    for (int n0 = 0; n0 < s.N; n0 += per_launch) {
        const int nb = std::min(per_launch, s.N - n0);
        prm.x = x + (size_t)n0 * img;
        prm.y = y + (size_t)n0 * s.K * prm.PQ;
        prm.M = nb * prm.PQ;
        prm.xbytes = (int)(nb * img * 4);
        rc = kConfigs[cfg].launch(prm, vec_w, st);
        if (rc != CNN_OK) return rc;
    }
    if (prm.splits > 1 && relu) {
        if (opt && opt->relu_left) {  // the consumer applies it
            *opt->relu_left = true;
            return CNN_OK;
        }
        return launch_relu(y, y, total, st);
    }
    return CNN_OK;
}

}  // namespace cnn
