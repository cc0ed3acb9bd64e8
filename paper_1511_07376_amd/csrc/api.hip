// libcnn C ABI: argument validation, dispatch to the kernels, and the network
// executor (a layer list run in order over two ping-pong activation buffers
// in a caller-provided workspace).
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "common.h"

namespace cnn {

namespace {
thread_local char g_err[512] = "";
}

int fail(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return status;
}

int check_launch(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(CNN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return CNN_OK;
}

KernelSpan*& current_span() {
    thread_local KernelSpan* span = nullptr;
    return span;
}

// Output extents are computed in 64 bits (a padding near INT_MAX must not
// wrap) and must fit an int.
int conv_out(int H, int W, int R, int S, int sh, int sw, int ph, int pw, int* P, int* Q) {
    if (H <= 0 || W <= 0) return fail(CNN_ERR_INVALID, "conv: input %dx%d is empty", H, W);
    if (R <= 0 || S <= 0) return fail(CNN_ERR_INVALID, "conv: kernel %dx%d", R, S);
    if (sh <= 0 || sw <= 0) return fail(CNN_ERR_INVALID, "conv: stride %dx%d", sh, sw);
    if (ph < 0 || pw < 0) return fail(CNN_ERR_INVALID, "conv: negative padding");
    const int64_t hp = (int64_t)H + 2 * (int64_t)ph, wp = (int64_t)W + 2 * (int64_t)pw;
    if (hp < R || wp < S)
        return fail(CNN_ERR_INVALID, "conv: kernel %dx%d larger than padded input %lldx%lld", R, S,
                    (long long)hp, (long long)wp);
    const int64_t p = (hp - R) / sh + 1, q = (wp - S) / sw + 1;
    if (p > INT32_MAX || q > INT32_MAX) return fail(CNN_ERR_UNSUPPORTED, "conv: output extent too large");
    *P = (int)p;
    *Q = (int)q;
    return CNN_OK;
}

namespace {
int64_t pool_extent(int64_t in, int64_t k, int64_t s, int64_t pad, int ceil_mode) {
    const int64_t span = in + 2 * pad - k;
    int64_t out = ceil_mode ? (span + s - 1) / s + 1 : span / s + 1;
    if (ceil_mode && (out - 1) * s >= in + pad) --out;  // window would start past the image
    return out;
}
}  // namespace

int pool_out(int H, int W, int kh, int kw, int sh, int sw, int ph, int pw, int ceil_mode, int* P,
             int* Q) {
    if (H <= 0 || W <= 0) return fail(CNN_ERR_INVALID, "pool: input %dx%d is empty", H, W);
    if (kh <= 0 || kw <= 0) return fail(CNN_ERR_INVALID, "pool: window %dx%d", kh, kw);
    if (sh <= 0 || sw <= 0) return fail(CNN_ERR_INVALID, "pool: stride %dx%d", sh, sw);
    if (ph < 0 || pw < 0 || ph >= kh || pw >= kw)
        return fail(CNN_ERR_INVALID, "pool: padding %dx%d must be >= 0 and below the window %dx%d",
                    ph, pw, kh, kw);
    if ((int64_t)H + 2 * (int64_t)ph < kh || (int64_t)W + 2 * (int64_t)pw < kw)
        return fail(CNN_ERR_INVALID, "pool: window larger than padded input");
    const int64_t p = pool_extent(H, kh, sh, ph, ceil_mode), q = pool_extent(W, kw, sw, pw, ceil_mode);
    if (p > INT32_MAX || q > INT32_MAX) return fail(CNN_ERR_UNSUPPORTED, "pool: output extent too large");
    *P = (int)p;
    *Q = (int)q;
    return CNN_OK;
}

namespace {

bool too_big(int64_t a, int64_t b, int64_t c = 1, int64_t d = 1) {
    // product of non-negative factors above the int32 element limit
    int64_t v = a;
    for (int64_t f : {b, c, d}) {
        if (f != 0 && v > kMaxElems / f) return true;
        v *= f;
    }
    return v > kMaxElems;
}

int check_conv(int N, int C, int H, int W, int K, int R, int S, int sh, int sw, int ph, int pw,
               int groups, ConvShape* s) {
    if (N < 0) return fail(CNN_ERR_INVALID, "conv: batch %d", N);
    if (C <= 0 || K <= 0) return fail(CNN_ERR_INVALID, "conv: channels C=%d K=%d", C, K);
    if (groups <= 0 || C % groups || K % groups)
        return fail(CNN_ERR_INVALID, "conv: groups=%d must divide C=%d and K=%d", groups, C, K);
    int P, Q;
    int rc = conv_out(H, W, R, S, sh, sw, ph, pw, &P, &Q);
    if (rc) return rc;
    if (too_big(N, C, H, W) || too_big(N, K, P, Q) || too_big(K, C / groups, R, S))
        return fail(CNN_ERR_UNSUPPORTED, "conv: a tensor exceeds 2^31-1 elements");
    *s = ConvShape{N, C, H, W, K, R, S, sh, sw, ph, pw, groups, P, Q};
    return CNN_OK;
}

int check_pool(int N, int C, int H, int W, int mode, int kh, int kw, int sh, int sw, int ph,
               int pw, int ceil_mode, PoolShape* s) {
    if (N < 0 || C <= 0) return fail(CNN_ERR_INVALID, "pool: N=%d C=%d", N, C);
    if (mode != CNN_POOL_MAX && mode != CNN_POOL_AVG)
        return fail(CNN_ERR_INVALID, "pool: mode %d", mode);
    int P, Q;
    int rc = pool_out(H, W, kh, kw, sh, sw, ph, pw, ceil_mode, &P, &Q);
    if (rc) return rc;
    if (too_big(N, C, H, W) || too_big(N, C, P, Q))  // padding can make the output the larger
        return fail(CNN_ERR_UNSUPPORTED, "pool: tensor exceeds 2^31-1 elements");
    *s = PoolShape{N, C, H, W, kh, kw, sh, sw, ph, pw, P, Q};
    return CNN_OK;
}

int check_lrn(int N, int C, int H, int W, int size) {
    if (N < 0 || C <= 0 || H <= 0 || W <= 0)
        return fail(CNN_ERR_INVALID, "lrn: shape %dx%dx%dx%d", N, C, H, W);
    if (size <= 0) return fail(CNN_ERR_INVALID, "lrn: size %d", size);
    if (size % 2 == 0) return fail(CNN_ERR_UNSUPPORTED, "lrn: even size %d", size);
    if (too_big(N, C, H, W)) return fail(CNN_ERR_UNSUPPORTED, "lrn: tensor exceeds 2^31-1 elements");
    return CNN_OK;
}

int check_softmax(int N, int C, int HW) {
    if (N < 0 || C <= 0 || HW <= 0) return fail(CNN_ERR_INVALID, "softmax: N=%d C=%d HW=%d", N, C, HW);
    if (too_big(N, C, HW)) return fail(CNN_ERR_UNSUPPORTED, "softmax: tensor exceeds 2^31-1 elements");
    return CNN_OK;
}

int check_fc(int N, int I, int O) {
    if (N < 0 || I <= 0 || O <= 0) return fail(CNN_ERR_INVALID, "fc: N=%d I=%d O=%d", N, I, O);
    if (too_big(N, I) || too_big(N, O) || too_big(O, I))
        return fail(CNN_ERR_UNSUPPORTED, "fc: tensor exceeds 2^31-1 elements");
    return CNN_OK;
}

// ------------------------------------------------------------------ networks
struct Plan {
    int type;
    int inC, inH, inW;     // input shape of the layer (per image)
    int outC, outH, outW;  // output shape
    int relu;              // ReLU executed inside this layer
    bool skipped;          // a RELU layer folded into its predecessor, or an LRN
                           // layer run inside the pooling layer after it
    int lrn_from;          // POOL: index of the LRN layer it runs first, or -1
    int opad_h, opad_w;    // POOL run with its LRN: the zero border its output
                           // planes get for the padded conv that reads them
    bool may_split;        // CONV, FC: some configuration splits the reduction
                           // across workgroups (room is kept for the output)
    bool split;            // ... and the one the launch will use does (the
                           // output must start as the bias)
    size_t split_off;      // may_split, not last: byte offset of its output in
                           // the split-output area of the workspace
    ConvShape conv;
    PoolShape pool;
};

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// need_weights: the net is about to run (shape queries take descriptors
// without parameters).  *split_bytes: size of the workspace area that holds
// the outputs of split-reduction conv and FC layers (other than the last
// layer), which are all set to their biases by one launch at the start of
// the pass.
// no_tune: the pass will not run the auto-tuner (shapes without a record take
// the heuristic).
int plan_net(const cnn_layer_desc* L, int n, int N, int C, int H, int W, Plan* plan,
             int64_t* max_elems, bool need_weights = true, size_t* split_bytes = nullptr,
             bool no_tune = false) {
    if (!L || n <= 0) return fail(CNN_ERR_INVALID, "net: no layers");
    if (N < 0 || C <= 0 || H <= 0 || W <= 0)
        return fail(CNN_ERR_INVALID, "net: input %dx%dx%dx%d", N, C, H, W);
    int c = C, h = H, w = W;
    int64_t mx = 0;
    int prev_exec = -1;  // index of the last executed (non-folded) layer
    for (int i = 0; i < n; ++i) {
        const cnn_layer_desc& d = L[i];
        Plan& p = plan[i];
        p = Plan{};
        p.lrn_from = -1;
        p.type = d.type;
        p.inC = c; p.inH = h; p.inW = w;
        int rc = CNN_OK;
        switch (d.type) {
            case CNN_LAYER_CONV: {
                if (need_weights && !d.weight)
                    return fail(CNN_ERR_INVALID, "net layer %d: conv without weights", i);
                if (d.in_channels != 0 && d.in_channels != c)
                    return fail(CNN_ERR_INVALID, "net layer %d: conv expects %d input channels, gets %d",
                                i, d.in_channels, c);
                rc = check_conv(N, c, h, w, d.out_channels, d.kernel_h, d.kernel_w, d.stride_h,
                                d.stride_w, d.pad_h, d.pad_w, d.groups, &p.conv);
                if (rc) return fail(rc, "net layer %d: %s", i, std::string(cnn_last_error()).c_str());
                // After an LRN + pooling kernel, the padding is written by that
                // kernel as a zero border around its output planes, and the
                // conv runs unpadded on the bordered planes: the gather then
                // needs no per-element padding test (3-5% on AlexNet's conv2
                // and conv3).
                if ((d.pad_h > 0 || d.pad_w > 0) && prev_exec >= 0 && plan[prev_exec].type == CNN_LAYER_POOL &&
                    plan[prev_exec].lrn_from >= 0) {
                    ConvShape bordered;
                    const int64_t hb64 = (int64_t)h + 2 * (int64_t)d.pad_h, wb64 = (int64_t)w + 2 * (int64_t)d.pad_w;
                    const int hb = (int)std::min<int64_t>(hb64, INT32_MAX), wb = (int)std::min<int64_t>(wb64, INT32_MAX);
                    // (the pooling kernel's bordered output planes stay below 2^24 elements)
                    if (hb64 < ((int64_t)1 << 24) && wb64 < ((int64_t)1 << 24) && hb64 * wb64 < ((int64_t)1 << 24) &&
                        check_conv(N, c, hb, wb, d.out_channels, d.kernel_h, d.kernel_w, d.stride_h,
                                   d.stride_w, 0, 0, d.groups, &bordered) == CNN_OK &&
                        bordered.P == p.conv.P && bordered.Q == p.conv.Q) {
                        p.conv = bordered;
                        plan[prev_exec].opad_h = d.pad_h;
                        plan[prev_exec].opad_w = d.pad_w;
                        mx = std::max<int64_t>(mx, (int64_t)N * c * hb * wb);
                    }
                }
                c = d.out_channels; h = p.conv.P; w = p.conv.Q;
                p.relu = d.fuse_relu != 0;
                if (N > 0) {
                    // the workspace does not depend on tuning: room for the output of
                    // any conv that some configuration splits; used when the
                    // configuration the launch will use (known unless it is still to
                    // be tuned) splits
                    for (int cfg = 0; cfg < conv2d_num_configs() && !p.may_split; ++cfg)
                        p.may_split = conv2d_splits(p.conv, cfg) > 1;
                    const int cfg = conv2d_planned_config(p.conv, no_tune);
                    p.split = cfg != -2 && conv2d_splits(p.conv, cfg) > 1;
                    p.may_split = p.may_split || p.split;
                }
                break;
            }
            case CNN_LAYER_FC: {
                if (need_weights && !d.weight)
                    return fail(CNN_ERR_INVALID, "net layer %d: fc without weights", i);
                const int64_t I = (int64_t)c * h * w;
                if (d.in_features != 0 && d.in_features != I)
                    return fail(CNN_ERR_INVALID, "net layer %d: fc expects %d inputs, gets %dx%dx%d = %lld",
                                i, d.in_features, c, h, w, (long long)I);
                if (I > kMaxElems) return fail(CNN_ERR_UNSUPPORTED, "net layer %d: fc input too large", i);
                rc = check_fc(N, (int)I, d.out_channels);
                if (rc) return fail(rc, "net layer %d: %s", i, std::string(cnn_last_error()).c_str());
                p.split = p.may_split = fc_splits(N, (int)I, d.out_channels) > 1;
                c = d.out_channels; h = 1; w = 1;
                p.relu = d.fuse_relu != 0;
                break;
            }
            case CNN_LAYER_POOL: {
                rc = check_pool(N, c, h, w, d.pool_mode, d.kernel_h, d.kernel_w, d.stride_h,
                                d.stride_w, d.pad_h, d.pad_w, d.ceil_mode, &p.pool);
                if (rc) return fail(rc, "net layer %d: %s", i, std::string(cnn_last_error()).c_str());
                if (d.pool_index && d.pool_mode != CNN_POOL_MAX)
                    return fail(CNN_ERR_INVALID, "net layer %d: indices requested for average pooling", i);
                // An LRN whose output only feeds this pooling layer runs inside it:
                // its output never goes to memory.
                if (prev_exec >= 0 && plan[prev_exec].type == CNN_LAYER_LRN &&
                    lrn_pool_fusable(p.pool, L[prev_exec].lrn_size)) {
                    plan[prev_exec].skipped = true;
                    p.lrn_from = prev_exec;
                }
                h = p.pool.P; w = p.pool.Q;
                p.relu = d.fuse_relu != 0;
                break;
            }
            case CNN_LAYER_LRN:
                rc = check_lrn(N, c, h, w, d.lrn_size);
                if (rc) return fail(rc, "net layer %d: %s", i, std::string(cnn_last_error()).c_str());
                break;
            case CNN_LAYER_SOFTMAX:
                rc = check_softmax(N, c, h * w);
                if (rc) return fail(rc, "net layer %d: %s", i, std::string(cnn_last_error()).c_str());
                break;
            case CNN_LAYER_RELU:
                // Embedded into the preceding conv / FC / pooling layer (Sec. 3.5).
                if (prev_exec >= 0 && (plan[prev_exec].type == CNN_LAYER_CONV ||
                                       plan[prev_exec].type == CNN_LAYER_FC ||
                                       plan[prev_exec].type == CNN_LAYER_POOL)) {
                    plan[prev_exec].relu = 1;
                    p.skipped = true;
                }
                break;
            default:
                return fail(CNN_ERR_INVALID, "net layer %d: unknown type %d", i, d.type);
        }
        p.outC = c; p.outH = h; p.outW = w;
        if (too_big(N, c, h, w)) return fail(CNN_ERR_UNSUPPORTED, "net layer %d: output too large", i);
        mx = std::max<int64_t>(mx, (int64_t)N * c * h * w);
        if (!p.skipped) prev_exec = i;
    }
    *max_elems = mx;
    int last = n - 1;
    while (last > 0 && plan[last].skipped) --last;
    size_t area = 0;
    for (int i = 0; i < n; ++i) {
        Plan& p = plan[i];
        if (p.may_split && !p.skipped && i != last) {
            p.split_off = area;
            area += align_up((size_t)N * p.outC * p.outH * p.outW * sizeof(float));
        }
    }
    if (split_bytes) *split_bytes = area;
    return CNN_OK;
}

// The kernel-timestamp span of layer i of a pass (nothing when starts is
// null): installed from construction to end().  end() reports whether the
// layer enqueued no kernel of its own (executed inside another one, or
// empty); run_net then records both of its events after the pass's last
// kernel, an interval of about zero, so that no record packet sits between
// two kernels of the pass.
class LayerSpan {
  public:
    LayerSpan(void* const* starts, void* const* stops, int i) {
        if (!starts) return;
        span_.start = reinterpret_cast<hipEvent_t>(starts[i]);
        span_.stop = reinterpret_cast<hipEvent_t>(stops[i]);
        current_span() = &span_;
        active_ = true;
    }
    ~LayerSpan() {
        if (active_) current_span() = nullptr;
    }
    LayerSpan(const LayerSpan&) = delete;
    LayerSpan& operator=(const LayerSpan&) = delete;
    int end(bool* empty) {
        *empty = false;
        if (!active_) return CNN_OK;
        current_span() = nullptr;
        active_ = false;
        *empty = !span_.started;
        return span_.started ? check_launch("kernel") : CNN_OK;
    }

  private:
    KernelSpan span_;
    bool active_ = false;
};

// Both events of every layer in `layers` (kernel-less layers), back to back.
int record_empty_spans(const std::vector<int>& layers, void* const* starts, void* const* stops, hipStream_t st) {
    for (int i : layers)
        if (hipEventRecord(reinterpret_cast<hipEvent_t>(starts[i]), st) != hipSuccess ||
            hipEventRecord(reinterpret_cast<hipEvent_t>(stops[i]), st) != hipSuccess)
            return check_launch("hipEventRecord");
    return CNN_OK;
}

// dumps (may be null): per layer, a device buffer that receives the layer's
// output as the layer list defines it (written[i] = 1), or nothing (written[i]
// = 0) for a RELU layer executed inside its predecessor, whose dump then holds
// the output after that ReLU.  An LRN run inside the pooling layer after it is
// also run on its own into its dump (the fused kernel never stores it).
// no_tune: never run the auto-tuner in this pass.
int run_net(const cnn_layer_desc* L, int n, const float* x, int N, int C, int H, int W, float* y,
            void* ws, size_t ws_bytes, void* const* events, hipStream_t st,
            float* const* dumps = nullptr, int* written = nullptr, bool no_tune = false,
            void* const* span_start = nullptr, void* const* span_stop = nullptr) {
    if (N != 0 && (!x || !y)) return fail(CNN_ERR_INVALID, "net: null input or output");
    if (n > 4096) return fail(CNN_ERR_UNSUPPORTED, "net: %d layers", n);
    std::vector<Plan> plan((size_t)std::max(n, 0));
    int64_t mx = 0;
    size_t split_bytes = 0;
    int rc = plan_net(L, n, N, C, H, W, plan.data(), &mx, true, &split_bytes, no_tune);
    if (rc) return rc;
    if (written)
        for (int i = 0; i < n; ++i) written[i] = 0;
    if (N == 0) {  // nothing to compute; still honour the event contract
        for (int i = 0; events && i <= n; ++i)
            if (hipEventRecord(reinterpret_cast<hipEvent_t>(events[i]), st) != hipSuccess)
                return check_launch("hipEventRecord");
        if (span_start) {
            std::vector<int> all((size_t)std::max(n, 0));
            for (int i = 0; i < n; ++i) all[(size_t)i] = i;
            return record_empty_spans(all, span_start, span_stop, st);
        }
        return CNN_OK;
    }
    const size_t half = align_up((size_t)mx * sizeof(float));
    if (!ws || ws_bytes < 2 * half + split_bytes)
        return fail(CNN_ERR_WORKSPACE, "net: workspace of %zu bytes, %zu needed", ws_bytes,
                    2 * half + split_bytes);
    if (reinterpret_cast<uintptr_t>(ws) % 16)
        return fail(CNN_ERR_INVALID, "net: workspace must be 16-byte aligned");
    float* buf[2] = {static_cast<float*>(ws),
                     reinterpret_cast<float*>(static_cast<char*>(ws) + half)};
    char* split_area = static_cast<char*>(ws) + 2 * half;

    int last = n - 1;
    while (last > 0 && plan[last].skipped) --last;

    // Every split-reduction output starts as its bias.  The pooling kernel
    // that runs just before the first such layer does the fills after its
    // own work (no launch of their own); otherwise one launch at the start
    // of the pass does them all.
    FillJobs host_fills;
    host_fills.n = 0;
    int fill_host = -1;
    {
        std::vector<BiasFill> fills;
        int first_split = -1;
        for (int i = 0; i < n; ++i) {
            const Plan& p = plan[i];
            if (!p.split || p.skipped) continue;
            if (first_split < 0) first_split = i;
            float* dst = i == last ? y : reinterpret_cast<float*>(split_area + p.split_off);
            fills.push_back(make_bias_fill(dst, L[i].bias, N, p.outC, p.outH * p.outW));
        }
        if (!fills.empty() && (int)fills.size() <= kMaxPoolFills) {
            int h = first_split - 1;
            while (h >= 0 && plan[h].skipped) --h;
            if (h >= 0 && plan[h].type == CNN_LAYER_POOL) {
                fill_host = h;
                host_fills.n = (int)fills.size();
                for (int j = 0; j < host_fills.n; ++j) host_fills.job[j] = fills[j];
            }
        }
        if (fill_host < 0) {
            rc = launch_bias_fills(fills.data(), (int)fills.size(), st);
            if (rc) return rc;
        }
    }

    const float* cur = x;
    int next_buf = 0;
    bool relu_pending = false;  // cur still needs the previous layer's ReLU
    std::vector<int> empty_spans;  // layers that enqueued no kernel (spans recorded at the end)
    for (int i = 0; i < n; ++i) {
        if (events) {
            if (hipEventRecord(reinterpret_cast<hipEvent_t>(events[i]), st) != hipSuccess)
                return check_launch("hipEventRecord");
        }
        LayerSpan span(span_start, span_stop, i);
        bool empty = false;
        const Plan& p = plan[i];
        if (p.skipped) {
            rc = span.end(&empty);
            if (rc) return rc;
            if (empty) empty_spans.push_back(i);
            continue;
        }
        const cnn_layer_desc& d = L[i];
        float* out = (i == last) ? y : buf[next_buf];
        if (p.split && i != last) out = reinterpret_cast<float*>(split_area + p.split_off);
        // A ReLU that a split-reduction layer would run as a pass of its own is
        // left to the next layer when that layer can take its input through a
        // ReLU as it reads it (conv, FC, pooling, LRN).
        int nx = i + 1;
        while (nx < n && plan[nx].skipped) ++nx;
        const bool next_takes_relu = nx < n && (plan[nx].type == CNN_LAYER_CONV || plan[nx].type == CNN_LAYER_FC ||
                                                plan[nx].type == CNN_LAYER_POOL || plan[nx].type == CNN_LAYER_LRN);
        bool* relu_left = next_takes_relu ? &relu_pending : nullptr;
        const bool relu_in = relu_pending;
        relu_pending = false;
        // an in-place ReLU or softmax keeps its buffer
        if ((p.type == CNN_LAYER_RELU || p.type == CNN_LAYER_SOFTMAX) && i != last && cur != x)
            out = const_cast<float*>(cur);
        switch (p.type) {
            case CNN_LAYER_CONV: {
                ConvOpts o;
                o.no_tune = no_tune;
                o.relu_in = relu_in;
                o.prefilled = p.split;
                o.relu_left = relu_left;
                rc = conv2d_dispatch(p.conv, cur, d.weight, d.bias, p.relu, out, st, &o);
                break;
            }
            case CNN_LAYER_FC:
                rc = launch_fc(cur, N, p.inC * p.inH * p.inW, d.weight, d.bias, p.outC, p.relu, out, st,
                               relu_in, relu_left, p.split);
                break;
            case CNN_LAYER_POOL: {
                const FillJobs* fj = i == fill_host ? &host_fills : nullptr;
                if (p.lrn_from >= 0) {  // cur is still the LRN's input
                    const cnn_layer_desc& ld = L[p.lrn_from];
                    if (dumps && dumps[p.lrn_from]) {
                        rc = launch_lrn(cur, N, p.inC, p.inH, p.inW, ld.lrn_size, ld.lrn_alpha, ld.lrn_beta,
                                        ld.lrn_k, dumps[p.lrn_from], st, relu_in);
                        if (rc) return fail(rc, "net layer %d: %s", p.lrn_from, std::string(cnn_last_error()).c_str());
                        if (written) written[p.lrn_from] = 1;
                    }
                    rc = launch_lrn_pool(p.pool, d.pool_mode, p.relu, ld.lrn_size, ld.lrn_alpha,
                                         ld.lrn_beta, ld.lrn_k, cur, out, d.pool_index, st, relu_in, fj,
                                         p.opad_h, p.opad_w);
                } else {
                    rc = launch_pool(p.pool, d.pool_mode, p.relu, cur, out, d.pool_index, st, relu_in, fj);
                }
                break;
            }
            case CNN_LAYER_LRN:
                rc = launch_lrn(cur, N, p.inC, p.inH, p.inW, d.lrn_size, d.lrn_alpha, d.lrn_beta,
                                d.lrn_k, out, st, relu_in);
                break;
            case CNN_LAYER_RELU:
                rc = launch_relu(cur, out, (int64_t)N * p.inC * p.inH * p.inW, st);
                break;
            case CNN_LAYER_SOFTMAX:
                rc = launch_softmax(cur, N, p.inC, p.inH * p.inW, out, st);
                break;
        }
        if (rc) return fail(rc, "net layer %d: %s", i, std::string(cnn_last_error()).c_str());
        rc = span.end(&empty);
        if (rc) return rc;
        if (empty) empty_spans.push_back(i);
        if (dumps && dumps[i]) {
            // the stored output without the zero border a pooling layer may give
            // it, and with a ReLU this layer left to the next one
            const int bh = p.type == CNN_LAYER_POOL ? p.opad_h : 0, bw = p.type == CNN_LAYER_POOL ? p.opad_w : 0;
            rc = launch_copy_planes(out, dumps[i], (int64_t)N * p.outC, p.outH, p.outW, bh, bw, relu_pending, st);
            if (rc) return fail(rc, "net layer %d: %s", i, std::string(cnn_last_error()).c_str());
            if (written) written[i] = 1;
        }
        if (out == buf[next_buf]) next_buf ^= 1;
        cur = out;
    }
    if (events) {
        if (hipEventRecord(reinterpret_cast<hipEvent_t>(events[n]), st) != hipSuccess)
            return check_launch("hipEventRecord");
    }
    if (span_start) return record_empty_spans(empty_spans, span_start, span_stop, st);
    return CNN_OK;
}

// ------------------------------------------------------------------ static scratch
// The workspace of cnn_net_fwd_noalloc: a device array of the library's own,
// one copy per GPU (allocated when the code object is loaded on that GPU and
// held until the process ends).  Host code never uses the array's name as an
// address: the device address of each GPU's copy is taken once, with that
// GPU current, and kept per device.
constexpr size_t kScratchBytes = CNN_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxScratchDevices] = {};

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// Device address of the current device's copy of `scratch`.
int scratch_of_current_device(void** addr) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return check_launch("hipGetDevice");
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(CNN_ERR_UNSUPPORTED, "net_fwd_noalloc: device %d beyond the %d supported", dev,
                    kMaxScratchDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(CNN_ERR_HIP, "net_fwd_noalloc: hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_addr[dev] = p;
    }
    *addr = g_scratch_addr[dev];
    return CNN_OK;
}

}  // namespace
}  // namespace cnn

using namespace cnn;

extern "C" {

int cnn_conv2d_out_shape(int H, int W, int R, int S, int sh, int sw, int ph, int pw, int* P, int* Q) {
    if (!P || !Q) return fail(CNN_ERR_INVALID, "conv_out_shape: null output pointer");
    return conv_out(H, W, R, S, sh, sw, ph, pw, P, Q);
}

int cnn_pool_out_shape(int H, int W, int kh, int kw, int sh, int sw, int ph, int pw, int ceil_mode,
                       int* P, int* Q) {
    if (!P || !Q) return fail(CNN_ERR_INVALID, "pool_out_shape: null output pointer");
    return pool_out(H, W, kh, kw, sh, sw, ph, pw, ceil_mode, P, Q);
}

int cnn_conv2d_fwd(const float* x, int N, int C, int H, int W, const float* w, int K, int R, int S,
                   const float* bias, int sh, int sw, int ph, int pw, int groups, int fuse_relu,
                   float* y, cnn_stream_t stream) {
    if ((N != 0 && (!x || !y)) || !w) return fail(CNN_ERR_INVALID, "conv: null x, w or y");
    ConvShape s;
    int rc = check_conv(N, C, H, W, K, R, S, sh, sw, ph, pw, groups, &s);
    if (rc) return rc;
    return conv2d_dispatch(s, x, w, bias, fuse_relu != 0, y, as_stream(stream));
}

int cnn_conv2d_fwd_config(const float* x, int N, int C, int H, int W, const float* w, int K, int R,
                          int S, const float* bias, int sh, int sw, int ph, int pw, int groups,
                          int fuse_relu, float* y, int config, cnn_stream_t stream) {
    if ((N != 0 && (!x || !y)) || !w) return fail(CNN_ERR_INVALID, "conv: null x, w or y");
    if (config < -1 || config >= conv2d_num_configs())
        return fail(CNN_ERR_INVALID, "conv: no configuration %d", config);
    ConvShape s;
    int rc = check_conv(N, C, H, W, K, R, S, sh, sw, ph, pw, groups, &s);
    if (rc) return rc;
    return launch_conv2d(s, x, w, bias, fuse_relu != 0, y, as_stream(stream), config);
}

int cnn_fc_fwd(const float* x, int N, int I, const float* w, const float* bias, int O, int fuse_relu,
               float* y, cnn_stream_t stream) {
    if ((N != 0 && (!x || !y)) || !w) return fail(CNN_ERR_INVALID, "fc: null x, w or y");
    int rc = check_fc(N, I, O);
    if (rc) return rc;
    return launch_fc(x, N, I, w, bias, O, fuse_relu != 0, y, as_stream(stream));
}

int cnn_fc_num_configs(void) { return fc_num_configs(); }

const char* cnn_fc_config_name(int i) { return fc_config_name(i); }

int cnn_fc_fwd_config(const float* x, int N, int I, const float* w, const float* bias, int O,
                      int fuse_relu, float* y, int config, cnn_stream_t stream) {
    if ((N != 0 && (!x || !y)) || !w) return fail(CNN_ERR_INVALID, "fc: null x, w or y");
    if (config < -1 || config >= fc_num_configs()) return fail(CNN_ERR_INVALID, "fc: no configuration %d", config);
    int rc = check_fc(N, I, O);
    if (rc) return rc;
    return launch_fc(x, N, I, w, bias, O, fuse_relu != 0, y, as_stream(stream), false, nullptr, false, config);
}

int cnn_pool_fwd(const float* x, int N, int C, int H, int W, int mode, int kh, int kw, int sh,
                 int sw, int ph, int pw, int ceil_mode, int fuse_relu, float* y, int32_t* idx,
                 cnn_stream_t stream) {
    if (N != 0 && (!x || !y)) return fail(CNN_ERR_INVALID, "pool: null x or y");
    PoolShape s;
    int rc = check_pool(N, C, H, W, mode, kh, kw, sh, sw, ph, pw, ceil_mode, &s);
    if (rc) return rc;
    if (idx && mode != CNN_POOL_MAX) return fail(CNN_ERR_INVALID, "pool: indices need max pooling");
    return launch_pool(s, mode, fuse_relu != 0, x, y, idx, as_stream(stream));
}

int cnn_lrn_fwd(const float* x, int N, int C, int H, int W, int size, float alpha, float beta,
                float k, float* y, cnn_stream_t stream) {
    if (N != 0 && (!x || !y)) return fail(CNN_ERR_INVALID, "lrn: null x or y");
    int rc = check_lrn(N, C, H, W, size);
    if (rc) return rc;
    return launch_lrn(x, N, C, H, W, size, alpha, beta, k, y, as_stream(stream));
}

int cnn_relu_fwd(const float* x, float* y, int64_t n, cnn_stream_t stream) {
    if (n != 0 && (!x || !y)) return fail(CNN_ERR_INVALID, "relu: null x or y");
    if (n < 0) return fail(CNN_ERR_INVALID, "relu: negative length");
    return launch_relu(x, y, n, as_stream(stream));
}

int cnn_softmax_fwd(const float* x, int N, int C, int HW, float* y, cnn_stream_t stream) {
    if (N != 0 && (!x || !y)) return fail(CNN_ERR_INVALID, "softmax: null x or y");
    int rc = check_softmax(N, C, HW);
    if (rc) return rc;
    if (x != y) {
        const size_t bytes = (size_t)N * C * HW * sizeof(float);
        const char* xb = reinterpret_cast<const char*>(x);
        const char* yb = reinterpret_cast<const char*>(y);
        if (xb < yb + bytes && yb < xb + bytes)
            return fail(CNN_ERR_INVALID, "softmax: x and y overlap without being equal");
    }
    return launch_softmax(x, N, C, HW, y, as_stream(stream));
}

int cnn_net_out_shape(const cnn_layer_desc* layers, int n_layers, int N, int C, int H, int W,
                      int* outC, int* outH, int* outW) {
    if (!outC || !outH || !outW) return fail(CNN_ERR_INVALID, "net_out_shape: null output pointer");
    if (n_layers > 4096) return fail(CNN_ERR_UNSUPPORTED, "net: %d layers", n_layers);
    std::vector<Plan> plan((size_t)std::max(n_layers, 0));
    int64_t mx;
    int rc = plan_net(layers, n_layers, N, C, H, W, plan.data(), &mx, false);
    if (rc) return rc;
    *outC = plan[n_layers - 1].outC;
    *outH = plan[n_layers - 1].outH;
    *outW = plan[n_layers - 1].outW;
    return CNN_OK;
}

size_t cnn_net_workspace_bytes(const cnn_layer_desc* layers, int n_layers, int N, int C, int H, int W) {
    if (n_layers > 4096 || n_layers <= 0) return 0;
    std::vector<Plan> plan((size_t)n_layers);
    int64_t mx;
    size_t split_bytes = 0;
    if (plan_net(layers, n_layers, N, C, H, W, plan.data(), &mx, false, &split_bytes)) return 0;
    return 2 * align_up((size_t)mx * sizeof(float)) + split_bytes;
}

int cnn_net_fwd(const cnn_layer_desc* layers, int n_layers, const float* x, int N, int C, int H,
                int W, float* y, void* ws, size_t ws_bytes, cnn_stream_t stream) {
    return run_net(layers, n_layers, x, N, C, H, W, y, ws, ws_bytes, nullptr, as_stream(stream));
}

int cnn_net_fwd_timed(const cnn_layer_desc* layers, int n_layers, const float* x, int N, int C,
                      int H, int W, float* y, void* ws, size_t ws_bytes, void* const* events,
                      cnn_stream_t stream) {
    if (!events) return fail(CNN_ERR_INVALID, "net_fwd_timed: null events");
    return run_net(layers, n_layers, x, N, C, H, W, y, ws, ws_bytes, events, as_stream(stream));
}

int cnn_net_fwd_kernel_timed(const cnn_layer_desc* layers, int n_layers, const float* x, int N, int C,
                             int H, int W, float* y, void* ws, size_t ws_bytes, void* const* start_events,
                             void* const* stop_events, cnn_stream_t stream) {
    if (!start_events || !stop_events) return fail(CNN_ERR_INVALID, "net_fwd_kernel_timed: null events");
    if (n_layers > 4096) return fail(CNN_ERR_UNSUPPORTED, "net: %d layers", n_layers);  // as run_net, before reading
    for (int i = 0; i < n_layers; ++i)
        if (!start_events[i] || !stop_events[i] || start_events[i] == stop_events[i])
            return fail(CNN_ERR_INVALID, "net_fwd_kernel_timed: layer %d needs two distinct events", i);
    return run_net(layers, n_layers, x, N, C, H, W, y, ws, ws_bytes, nullptr, as_stream(stream), nullptr,
                   nullptr, false, start_events, stop_events);
}

int cnn_net_fwd_noalloc(const cnn_layer_desc* layers, int n_layers, const float* x, int N, int C, int H,
                        int W, float* y, cnn_stream_t stream) {
    if (n_layers > 4096) return fail(CNN_ERR_UNSUPPORTED, "net: %d layers", n_layers);
    std::vector<Plan> plan((size_t)std::max(n_layers, 0));
    int64_t mx = 0;
    size_t split_bytes = 0;
    int rc = plan_net(layers, n_layers, N, C, H, W, plan.data(), &mx, true, &split_bytes, true);
    if (rc) return rc;
    const size_t need = 2 * align_up((size_t)mx * sizeof(float)) + split_bytes;
    if (need > kScratchBytes)
        return fail(CNN_ERR_WORKSPACE,
                    "net_fwd_noalloc: this input needs %zu bytes of workspace, the static scratch holds %zu "
                    "(use cnn_net_fwd with a workspace of cnn_net_workspace_bytes())",
                    need, kScratchBytes);
    void* ws = nullptr;
    if (N > 0) {
        rc = scratch_of_current_device(&ws);
        if (rc) return rc;
    }
    return run_net(layers, n_layers, x, N, C, H, W, y, ws, kScratchBytes, nullptr, as_stream(stream), nullptr,
                   nullptr, true);
}

int cnn_net_fwd_dump(const cnn_layer_desc* layers, int n_layers, const float* x, int N, int C, int H,
                     int W, float* y, void* ws, size_t ws_bytes, float* const* dumps, int* written,
                     cnn_stream_t stream) {
    if (!dumps) return fail(CNN_ERR_INVALID, "net_fwd_dump: null dump array");
    return run_net(layers, n_layers, x, N, C, H, W, y, ws, ws_bytes, nullptr, as_stream(stream), dumps,
                   written);
}

}  // extern "C"

struct cnn_net_graph {
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;  // null for an empty batch
};

extern "C" {

int cnn_net_graph_create(const cnn_layer_desc* layers, int n_layers, const float* x, int N, int C,
                         int H, int W, float* y, void* ws, size_t ws_bytes, cnn_net_graph** graph) {
    if (!graph) return fail(CNN_ERR_INVALID, "net_graph: null output handle");
    *graph = nullptr;
    auto* g = new (std::nothrow) cnn_net_graph;
    if (!g) return fail(CNN_ERR_INVALID, "net_graph: out of host memory");
    if (N == 0) {  // validate only: the replay does nothing
        std::vector<Plan> plan((size_t)std::max(n_layers, 0));
        int64_t mx;
        if (n_layers > 4096) { delete g; return fail(CNN_ERR_UNSUPPORTED, "net: %d layers", n_layers); }
        const int rc = plan_net(layers, n_layers, N, C, H, W, plan.data(), &mx);
        if (rc) { delete g; return rc; }
        *graph = g;
        return CNN_OK;
    }
    hipStream_t cs;
    if (hipStreamCreateWithFlags(&cs, hipStreamNonBlocking) != hipSuccess) {
        delete g;
        return check_launch("hipStreamCreateWithFlags");
    }
    int rc = CNN_OK;
    if (hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal) != hipSuccess) {
        rc = check_launch("hipStreamBeginCapture");
    } else {
        rc = run_net(layers, n_layers, x, N, C, H, W, y, ws, ws_bytes, nullptr, cs);
        const hipError_t e = hipStreamEndCapture(cs, &g->graph);
        if (rc == CNN_OK && e != hipSuccess) rc = fail(CNN_ERR_HIP, "hipStreamEndCapture: %s", hipGetErrorString(e));
    }
    if (rc == CNN_OK && hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0) != hipSuccess)
        rc = check_launch("hipGraphInstantiate");
    (void)hipStreamDestroy(cs);
    if (rc != CNN_OK) {
        if (g->graph) (void)hipGraphDestroy(g->graph);
        delete g;
        return rc;
    }
    *graph = g;
    return CNN_OK;
}

int cnn_net_graph_launch(cnn_net_graph* graph, cnn_stream_t stream) {
    if (!graph) return fail(CNN_ERR_INVALID, "net_graph: null handle");
    if (!graph->exec) return CNN_OK;
    if (hipGraphLaunch(graph->exec, as_stream(stream)) != hipSuccess) return check_launch("hipGraphLaunch");
    return CNN_OK;
}

int cnn_net_graph_destroy(cnn_net_graph* graph) {
    if (!graph) return CNN_OK;
    int rc = CNN_OK;
    if (graph->exec && hipGraphExecDestroy(graph->exec) != hipSuccess) rc = check_launch("hipGraphExecDestroy");
    if (graph->graph && hipGraphDestroy(graph->graph) != hipSuccess) rc = check_launch("hipGraphDestroy");
    delete graph;
    return rc;
}

const char* cnn_last_error(void) { return g_err; }

const char* cnn_version(void) { return "libcnn 0.1 gfx950"; }

}  // extern "C"
