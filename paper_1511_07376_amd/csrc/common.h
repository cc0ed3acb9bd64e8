// Internal declarations shared by the libcnn translation units.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/cnn.h"

namespace cnn {

// Records a thread-local error message and returns `status`.
int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Checks hipGetLastError() after launches; CNN_OK or CNN_ERR_HIP.
int check_launch(const char* what);

inline hipStream_t as_stream(cnn_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

// Timing of a layer by its kernels' own timestamps.  While a span is installed
// on the calling thread, the first kernel the library enqueues gives `start`
// that kernel's start time and every kernel gives `stop` its end time (the
// last one's stands), so stop - start covers the layer's kernels and nothing
// else: no marker packet of its own enters the stream.
struct KernelSpan {
    hipEvent_t start = nullptr, stop = nullptr;
    bool started = false;
};
KernelSpan*& current_span();

// Every kernel of the library is enqueued through this.
template <typename F, typename... Args>
inline void enqueue(F kernel, const dim3& grid, const dim3& block, uint32_t shm, hipStream_t st, Args... args) {
    KernelSpan* s = current_span();
    if (!s) {
        hipLaunchKernelGGL(kernel, grid, block, shm, st, args...);
        return;
    }
    hipExtLaunchKernelGGL(kernel, grid, block, shm, st, s->started ? nullptr : s->start, s->stop, 0u, args...);
    s->started = true;
}

// No span is installed during its lifetime (the auto-tuner's timing runs).
class SpanPause {
  public:
    SpanPause() : saved_(current_span()) { current_span() = nullptr; }
    ~SpanPause() { current_span() = saved_; }
    SpanPause(const SpanPause&) = delete;
    SpanPause& operator=(const SpanPause&) = delete;

  private:
    KernelSpan* saved_;
};

// Division by a runtime constant through a multiply-high (exact for n < 2^31):
// the unsigned method of Granlund and Montgomery, "Division by invariant
// integers using multiplication" (PLDI 1994), with l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1, so that n / d = (mulhi(m, n) + n) >> l.
// A divisor of 0 is taken as 1 (only for launches that do no work).
struct FastDiv {
    unsigned m, l;
};
inline FastDiv make_fastdiv(unsigned d) {
    if (d == 0) d = 1;
    unsigned l = 0;
    while ((1u << l) < d) ++l;
    const uint64_t m = ((((uint64_t)1 << l) - d) << 32) / d + 1;
    return FastDiv{(unsigned)m, l};
}
__device__ inline unsigned fdiv(unsigned n, FastDiv f) { return (__umulhi(f.m, n) + n) >> f.l; }

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Largest element count a tensor may have (offsets inside kernels are int32).
constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;

struct ConvShape {
    int N, C, H, W, K, R, S, sh, sw, ph, pw, G, P, Q;
};

struct PoolShape {
    int N, C, H, W, kh, kw, sh, sw, ph, pw, P, Q;
};

// Shape helpers (return CNN_OK or an error status with a message).
int conv_out(int H, int W, int R, int S, int sh, int sw, int ph, int pw, int* P, int* Q);
int pool_out(int H, int W, int kh, int kw, int sh, int sw, int ph, int pw, int ceil_mode,
             int* P, int* Q);

// Launchers: arguments already validated; they enqueue and return CNN_OK or
// CNN_ERR_HIP.
// Options of a convolution run inside a network:
//   relu_in   take the input through a ReLU as it is read (the producer left
//             its ReLU to this layer);
//   prefilled y already holds the bias (only with a split reduction);
//   relu_left non-null: a ReLU that would need a pass of its own (split
//             reduction) is skipped and *relu_left set, for the consumer.
//   no_tune   never run the auto-tuner for this call (a shape without a
//             record takes the heuristic), as for a caller that must not
//             allocate or synchronise.
struct ConvOpts {
    bool relu_in = false;
    bool prefilled = false;
    bool* relu_left = nullptr;
    bool no_tune = false;
};
// cfg: index into the convolution configuration table, or -1 for the
// built-in heuristic.
int launch_conv2d(const ConvShape& s, const float* x, const float* w, const float* bias,
                  int relu, float* y, hipStream_t st, int cfg, const ConvOpts* opt = nullptr);
int conv2d_num_configs();
const char* conv2d_config_name(int i);
// Reduction splits configuration cfg (-1: heuristic) uses for this shape.
int conv2d_splits(const ConvShape& s, int cfg);
// The built-in heuristic's configuration for this shape (-1 if none applies).
int conv2d_heuristic_config(const ConvShape& s);
// Convolution with the tuned configuration for this shape (auto-tuning it
// first when auto-tuning is on and the shape is new).
int conv2d_dispatch(const ConvShape& s, const float* x, const float* w, const float* bias,
                    int relu, float* y, hipStream_t st, const ConvOpts* opt = nullptr);
// The configuration conv2d_dispatch would use now: the tuned one, else the
// heuristic (-1); -2 when the shape would be auto-tuned first (never with
// no_tune).
int conv2d_planned_config(const ConvShape& s, bool no_tune = false);
// relu_in: apply a ReLU to x as it is read.  relu_left non-null: when the
// layer's ReLU would need a pass of its own (split reduction), skip it and set
// *relu_left, so that the caller can fold it into the next layer's input.
// prefilled: y already holds the bias (see fc_splits, launch_bias_fills).
// config: an FC kernel configuration (0 <= config < fc_num_configs()), or -1
// for the built-in choice.
int launch_fc(const float* x, int N, int I, const float* w, const float* bias, int O, int relu,
              float* y, hipStream_t st, bool relu_in = false, bool* relu_left = nullptr,
              bool prefilled = false, int config = -1);
int fc_num_configs();
const char* fc_config_name(int i);
// Reduction splits of the built-in choice for this shape (launch_fc with
// config -1); above 1 its output must start as the bias (launch_fc fills it
// unless told it is prefilled).  Batches of at most kGemvMaxN images take an
// unsplit matrix-vector kernel.
constexpr int kGemvMaxN = 2;
int fc_splits(int N, int I, int O);
// y_j[n][o][i] = bias_j[o] (or 0), i < inner, for several layer outputs
// (FC: inner = 1; conv NCHW: inner = P*Q), in one launch per kMaxBiasFills
// jobs.
constexpr int kMaxBiasFills = 8;
// A pooling kernel carries at most this many, so that its parameter block
// stays within the size it had before the fills were added (a block 190 bytes
// larger made the LRN + pooling kernels of AlexNet at batch 64 0.5 us slower
// each, fills or not).  AlexNet at batch 16 has 6 split layers.
constexpr int kMaxPoolFills = 6;
struct BiasFill {
    float* y;
    const float* bias;
    int total;             // N * O * inner elements, below 2^31
    int O;
    FastDiv f_inner, f_o;  // division by inner and by O
};
inline BiasFill make_bias_fill(float* y, const float* bias, int N, int O, int inner) {
    return BiasFill{y, bias, N * O * inner, O, make_fastdiv(inner), make_fastdiv(O)};
}
int launch_bias_fills(const BiasFill* jobs, int n, hipStream_t st);
// Up to CAP of them, as a kernel argument: bias_fill_multi runs up to
// kMaxBiasFills on their own, and a pooling kernel up to kMaxPoolFills after
// its own work (fills argument of launch_pool / launch_lrn_pool), which saves
// the network executor a launch.
template <int CAP>
struct FillJobsOf {
    BiasFill job[CAP];
    int n;
};
using FillJobs = FillJobsOf<kMaxPoolFills>;
// relu_x (pooling, LRN): take the input through a ReLU as it is read.
// fills: bias fills the kernel also performs (NULL: none).
int launch_pool(const PoolShape& s, int mode, int relu, const float* x, float* y, int32_t* idx,
                hipStream_t st, bool relu_x = false, const FillJobs* fills = nullptr);
int launch_lrn(const float* x, int N, int C, int H, int W, int size, float alpha, float beta,
               float k, float* y, hipStream_t st, bool relu_x = false);
int launch_relu(const float* x, float* y, int64_t n, hipStream_t st);
// LRN (across channels, odd size) followed by pooling of its output, in one
// kernel; s is the pooling shape (its input is the LRN's shape).  Only where
// lrn_pool_fusable() holds.  opad_h, opad_w > 0: y holds each output plane
// inside a zero border of that width ((P + 2 opad_h) x (Q + 2 opad_w) per
// plane), the input layout of a padded convolution run as unpadded; idx keeps
// the plain P x Q layout.
bool lrn_pool_fusable(const PoolShape& s, int size);
int launch_lrn_pool(const PoolShape& s, int mode, int relu, int size, float alpha, float beta, float k,
                    const float* x, float* y, int32_t* idx, hipStream_t st, bool relu_x = false,
                    const FillJobs* fills = nullptr, int opad_h = 0, int opad_w = 0);
int launch_softmax(const float* x, int N, int C, int HW, float* y, hipStream_t st);
// dst [planes][P][Q] = the inner P x Q of src's planes of (P + 2 bh) x
// (Q + 2 bw), through a ReLU when relu is set.
int launch_copy_planes(const float* src, float* dst, int64_t planes, int P, int Q, int bh, int bw,
                       bool relu, hipStream_t st);

}  // namespace cnn
