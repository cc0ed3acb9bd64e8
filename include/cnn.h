/*
 * cnn.h -- C ABI of libcnn, the gfx950 (MI355X) forward pass of trained CNNs.
 *
 * The layer set is the one the paper's library executes: convolution, max and
 * mean pooling, fully connected, ReLU and local response normalization
 * (Sec. 3.1), chained into networks that run on one image or a batch
 * (Sec. 3.3, the compute() call), with ReLU embedded into the preceding
 * layer (Sec. 3.5).  The paper gives no formulas; each entry point states
 * the definition it computes.
 *
 * Conventions for every entry point:
 *  - Tensors are fp32, NCHW, row-major, contiguous, in DEVICE memory,
 *    allocated and owned by the caller.  The library allocates nothing.
 *  - Calls are asynchronous: argument checks run on the host first and a
 *    negative status means nothing was enqueued; on CNN_OK the kernels are
 *    enqueued on `stream` (a hipStream_t; NULL = the null stream) and the
 *    caller synchronises.
 *  - Input and output buffers must not overlap, except that cnn_relu_fwd
 *    and cnn_softmax_fwd allow y == x.  A pointer to a tensor with no elements (batch N = 0,
 *    length n = 0) may be NULL; such a call validates and enqueues nothing.
 *  - No exception or abort crosses the ABI.  cnn_last_error() returns a
 *    thread-local message describing the last non-OK status of this thread.
 *  - Sizes are int (each tensor must hold fewer than 2^31 elements).
 */
#ifndef CNN_H
#define CNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum cnn_status {
    CNN_OK = 0,
    CNN_ERR_INVALID = -1,     /* bad argument: null pointer, bad size, inconsistent shapes */
    CNN_ERR_UNSUPPORTED = -2, /* well-formed but outside what the kernels implement */
    CNN_ERR_HIP = -3,         /* the HIP runtime reported an error at launch */
    CNN_ERR_WORKSPACE = -4    /* workspace missing or smaller than required */
} cnn_status;

typedef void* cnn_stream_t; /* hipStream_t */

/* Convolution output size, floor rule: P = (H + 2*ph - R) / sh + 1,
 * Q = (W + 2*pw - S) / sw + 1.  Requires H + 2*ph >= R, W + 2*pw >= S,
 * strides >= 1, pads >= 0. */
int cnn_conv2d_out_shape(int H, int W, int R, int S, int sh, int sw,
                         int ph, int pw, int* P, int* Q);

/* Pooling output size.  ceil_mode = 1: P = ceil((H + 2*ph - kh) / sh) + 1,
 * then one less if that last window would start at or past H + ph (so that
 * every window overlaps the image); ceil_mode = 0: floor instead of ceil.
 * Requires 0 <= ph < kh and 0 <= pw < kw. */
int cnn_pool_out_shape(int H, int W, int kh, int kw, int sh, int sw,
                       int ph, int pw, int ceil_mode, int* P, int* Q);

/* Convolution layer (Sec. 3.1; computed on the GPU, Sec. 3.5): grouped 2-D
 * cross-correlation (no kernel flip) with stride, zero padding and bias,
 *   y[n,k,p,q] = b[k] + sum_{c < C/G, r < R, s < S}
 *                x[n, g*C/G + c, p*sh - ph + r, q*sw - pw + s] * w[k,c,r,s]
 * where g = k / (K/G) and x is zero outside the image.
 *   x    [N][C][H][W]      w [K][C/G][R][S]      bias [K] or NULL
 *   y    [N][K][P][Q]      (P, Q from cnn_conv2d_out_shape)
 * groups must divide C and K.  fuse_relu = 1 applies y = max(y, 0) in the
 * same kernel (a Conv+ReLU layer).  When the output has too few tiles to
 * occupy the GPU (small batches), the reduction is split across workgroups:
 * y is first set to the bias, the partial sums are added with fp32 atomics
 * and the ReLU runs as a separate pass; the summation order, and so the last
 * bits of y, may then differ from call to call.  Errors: CNN_ERR_INVALID for
 * null x/w/y, non-positive sizes or bad shapes. */
int cnn_conv2d_fwd(const float* x, int N, int C, int H, int W,
                   const float* w, int K, int R, int S, const float* bias,
                   int sh, int sw, int ph, int pw, int groups, int fuse_relu,
                   float* y, cnn_stream_t stream);

/* ---------------------------------------------------------------- tuning
 * The paper's library has tuning parameters that set the work per GPU thread
 * and per SIMD unit, and an optional auto-tuner that times predefined
 * scenarios on first launch and keeps the fastest (Sec. 3.6).  Here the
 * tuning parameter is the convolution kernel's tile configuration.
 */

/* Number of convolution tile configurations in this build, and a readable
 * name for configuration i (NULL when out of range). */
int cnn_conv2d_num_configs(void);
const char* cnn_conv2d_config_name(int i);

/* cnn_conv2d_fwd with an explicit tile configuration: 0 <= config <
 * cnn_conv2d_num_configs(), or -1 for the built-in heuristic (ignoring any
 * tuned entry).  Every configuration computes the same function. */
int cnn_conv2d_fwd_config(const float* x, int N, int C, int H, int W,
                          const float* w, int K, int R, int S, const float* bias,
                          int sh, int sw, int ph, int pw, int groups, int fuse_relu,
                          float* y, int config, cnn_stream_t stream);

/* Auto-tuning switch (process-wide; default 0 = off).  With 1, the first
 * cnn_conv2d_fwd / cnn_net_fwd call that meets a new convolution shape runs
 * every configuration on that call's own buffers, synchronising its stream
 * (not while the stream is being captured), and records the fastest for the
 * shape; the call then returns normally with the result of the chosen
 * configuration.  Later calls of the shape use the record, tuning on or off. */
int cnn_set_autotune(int mode);

/* The tuning records as text, one line per shape:
 *   "N C H W K R S sh sw ph pw G config\n".
 * Writes at most cap bytes (NUL-terminated) to buf when buf is not NULL and
 * returns the size the whole text needs, NUL included. */
size_t cnn_tuning_export(char* buf, size_t cap);

/* Adds records in the export format (lines starting with '#' are skipped);
 * returns the number of records read, or CNN_ERR_INVALID on a malformed line
 * (records before it are kept). */
int cnn_tuning_import(const char* text);

/* Forgets every tuning record. */
int cnn_tuning_clear(void);

/* Fully-connected layer (Sec. 3.1; a matrix-vector product per image,
 * Sec. 3.5): y[n,o] = b[o] + sum_i x[n,i] * w[o,i].
 *   x [N][I] (an NCHW tensor flattened: i = c*H*W + h*W + w)
 *   w [O][I]   bias [O] or NULL   y [N][O]
 * fuse_relu = 1 applies y = max(y, 0) (an FC+ReLU layer).  For N >= 1 the
 * result is the same for every batch split; when the reduction is split
 * across workgroups the summation order is not fixed run to run. */
int cnn_fc_fwd(const float* x, int N, int I, const float* w,
               const float* bias, int O, int fuse_relu, float* y,
               cnn_stream_t stream);

/* Number of FC kernel configurations in this build, and a readable name for
 * configuration i (NULL when out of range). */
int cnn_fc_num_configs(void);
const char* cnn_fc_config_name(int i);

/* cnn_fc_fwd (Sec. 3.1) with an explicit kernel configuration: 0 <= config <
 * cnn_fc_num_configs(), or -1 for the built-in choice.  Every configuration
 * computes the same function; CNN_ERR_UNSUPPORTED when the configuration
 * does not take the shape (a batch above its limit, or, for the ones that
 * load 128 bits at a time, I not a multiple of 4 or x, w not 16-byte
 * aligned).  Same arguments and ownership as cnn_fc_fwd otherwise. */
int cnn_fc_fwd_config(const float* x, int N, int I, const float* w,
                      const float* bias, int O, int fuse_relu, float* y,
                      int config, cnn_stream_t stream);

typedef enum cnn_pool_mode { CNN_POOL_MAX = 0, CNN_POOL_AVG = 1 } cnn_pool_mode;

/* Max / mean pooling layer (Sec. 3.1).  Window (p, q) covers rows
 * [p*sh - ph, p*sh - ph + kh) and columns [q*sw - pw, q*sw - pw + kw),
 * clipped to the image.
 *   MAX: y = the largest element; idx (optional, int32 [N][C][P][Q]) receives
 *        h*W + w of the FIRST largest element in row-major order.
 *   AVG: y = (sum of the clipped window) / (window area clipped to the padded
 *        extent [-ph, H + ph) x [-pw, W + pw)).
 * fuse_relu = 1 applies y = max(y, 0) after pooling (a Pooling+ReLU layer);
 * the index stays that of the pre-ReLU maximum.  idx must be NULL for AVG.
 * Inputs must be finite (NaN ordering is not defined). */
int cnn_pool_fwd(const float* x, int N, int C, int H, int W, int mode,
                 int kh, int kw, int sh, int sw, int ph, int pw, int ceil_mode,
                 int fuse_relu, float* y, int32_t* idx, cnn_stream_t stream);

/* Local response normalization across channels (Sec. 3.1; AlexNet rows of
 * the layer-setup table, Sec. 4):
 *   y[n,c,h,w] = x[n,c,h,w] * (k + alpha/size * sum_{c'} x[n,c',h,w]^2)^(-beta)
 * with c' over [c - size/2, c + size/2] clipped to [0, C).  size must be odd
 * (CNN_ERR_UNSUPPORTED otherwise). */
int cnn_lrn_fwd(const float* x, int N, int C, int H, int W, int size,
                float alpha, float beta, float k, float* y, cnn_stream_t stream);

/* ReLU layer (Sec. 3.1): y[i] = x[i] > 0 ? x[i] : +0.0f for i < n.
 * y == x (in place) is allowed. */
int cnn_relu_fwd(const float* x, float* y, int64_t n, cnn_stream_t stream);

/* Softmax layer (Sec. 3.1), across channels of x viewed as [N][C][HW]
 * (HW = H*W of an NCHW tensor, 1 after a fully connected layer):
 *   y[n,c,i] = exp(x[n,c,i] - m) / sum_{c'} exp(x[n,c',i] - m),
 *   m = max_{c'} x[n,c',i].
 * y == x (in place) is allowed; other overlaps are CNN_ERR_INVALID.  Inputs
 * must be finite (NaN / infinity give unspecified results). */
int cnn_softmax_fwd(const float* x, int N, int C, int HW, float* y, cnn_stream_t stream);

/* ---------------------------------------------------------------- networks
 * A network is an array of layer descriptors executed in order (the paper's
 * NetFile layer list, Sec. 3.2, and compute(), Sec. 3.3).  Parameters are
 * caller-owned device buffers that stay resident between calls.
 */
typedef enum cnn_layer_type {
    CNN_LAYER_CONV = 0,
    CNN_LAYER_FC = 1,
    CNN_LAYER_POOL = 2,
    CNN_LAYER_LRN = 3,
    CNN_LAYER_RELU = 4,
    CNN_LAYER_SOFTMAX = 5
} cnn_layer_type;

typedef struct cnn_layer_desc {
    int32_t type;          /* cnn_layer_type */
    int32_t out_channels;  /* CONV: K; FC: O */
    int32_t kernel_h;      /* CONV: R; POOL: kh */
    int32_t kernel_w;      /* CONV: S; POOL: kw */
    int32_t stride_h;      /* CONV, POOL */
    int32_t stride_w;
    int32_t pad_h;         /* CONV, POOL */
    int32_t pad_w;
    int32_t groups;        /* CONV (>= 1) */
    int32_t pool_mode;     /* POOL: cnn_pool_mode */
    int32_t ceil_mode;     /* POOL */
    int32_t fuse_relu;     /* CONV, FC, POOL: ReLU after the layer */
    int32_t lrn_size;      /* LRN */
    float lrn_alpha;       /* LRN */
    float lrn_beta;        /* LRN */
    float lrn_k;           /* LRN */
    int32_t in_channels;   /* CONV: expected input channels C (0 = not checked) */
    int32_t in_features;   /* FC: expected C*H*W of its input (0 = not checked) */
    const float* weight;   /* CONV: [K][C/G][R][S]; FC: [O][I] */
    const float* bias;     /* CONV: [K]; FC: [O]; or NULL */
    int32_t* pool_index;   /* POOL MAX: optional int32 [N][C][P][Q] output */
} cnn_layer_desc;

/* Output shape of the network for an N x C x H x W input (outC x outH x outW
 * per image; FC layers give outH = outW = 1).  CNN_ERR_INVALID /
 * CNN_ERR_UNSUPPORTED describe the first bad layer.  Weight pointers are not
 * needed here (nor by cnn_net_workspace_bytes). */
int cnn_net_out_shape(const cnn_layer_desc* layers, int n_layers, int N, int C,
                      int H, int W, int* outC, int* outH, int* outW);

/* Device workspace cnn_net_fwd needs for this input: two activation buffers
 * of the largest intermediate tensor, each 256-byte aligned (a pooling layer
 * run with its LRN writes its planes inside the zero border of a padded CONV
 * layer that reads them, which then runs unpadded: such planes count with
 * their border), plus room for
 * the outputs of the conv and FC layers whose reduction may be split across
 * workgroups (small outputs, e.g. at batch 1; they are set to their biases
 * together, by the pooling kernel that runs just before the first of them,
 * or else by one launch at the start of a pass).  The size does not depend
 * on tuning.  0 on error. */
size_t cnn_net_workspace_bytes(const cnn_layer_desc* layers, int n_layers,
                               int N, int C, int H, int W);

/* Runs the network on x [N][C][H][W] and writes the last layer's output to y
 * ([N][outC][outH][outW]).  ws is caller-owned device memory of at least
 * cnn_net_workspace_bytes(); intermediates live there.  A RELU layer that
 * follows a CONV, FC or POOL layer is executed inside that layer (Sec. 3.5);
 * an LRN layer followed by a POOL layer runs inside that pooling kernel (its
 * output never goes to memory; the values equal those of the two layers run
 * separately, bit for bit); other RELU layers and SOFTMAX layers run in
 * place.  A SOFTMAX layer uses
 * only the type field.  Every layer is validated before the first launch;
 * a list of more than 4096 layers gives CNN_ERR_UNSUPPORTED. */
int cnn_net_fwd(const cnn_layer_desc* layers, int n_layers, const float* x,
                int N, int C, int H, int W, float* y, void* ws, size_t ws_bytes,
                cnn_stream_t stream);

/* As cnn_net_fwd, and records events[i] (hipEvent_t) on the stream before
 * layer i and events[n_layers] after the last one, so that the caller can
 * time each layer (the paper times whole networks and the heaviest conv
 * layer separately, Sec. 4.2).  A RELU layer executed inside its predecessor,
 * and an LRN layer executed inside the pooling layer after it, get an empty
 * interval; the bias fills of split layers count in the interval of the
 * pooling layer that performs them. */
int cnn_net_fwd_timed(const cnn_layer_desc* layers, int n_layers, const float* x,
                      int N, int C, int H, int W, float* y, void* ws,
                      size_t ws_bytes, void* const* events, cnn_stream_t stream);

/* As cnn_net_fwd, and times every layer by its kernels' own timestamps (the
 * paper times whole networks and the heaviest conv layer separately,
 * Sec. 4.2): start_events[i] and stop_events[i] (hipEvent_t, created by the
 * caller, two distinct events per layer, n_layers of each) receive the start
 * of layer i's first kernel and the end of its last one, so that
 * hipEventElapsedTime(start_events[i], stop_events[i]) is the layer's
 * kernel time, with no marker packets between the layers (unlike
 * cnn_net_fwd_timed, whose event records add a few microseconds to each
 * interval).
 *   - A layer that launches no kernel of its own (a RELU run inside its
 *     predecessor, an LRN run inside the pooling layer after it) gets both
 *     events recorded back to back after the pass's last kernel: an
 *     interval of about zero, outside every other layer's span.
 *   - The bias fills of split layers count in the interval of the pooling
 *     layer that performs them; when no pooling layer can, their one launch
 *     at the start of the pass is in no interval.
 *   - A conv layer that the auto-tuner times during this pass counts only
 *     its final launch, not the candidates' runs.
 *   - Null arrays, or a null or repeated event for a layer, give
 *     CNN_ERR_INVALID before any work is enqueued. */
int cnn_net_fwd_kernel_timed(const cnn_layer_desc* layers, int n_layers,
                             const float* x, int N, int C, int H, int W,
                             float* y, void* ws, size_t ws_bytes,
                             void* const* start_events, void* const* stop_events,
                             cnn_stream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): cnn_net_fwd
 * with the library's own static device scratch as the workspace, of
 * CNN_NOALLOC_SCRATCH_BYTES per GPU (256 MiB: AlexNet-shaped networks up to
 * batch 64, LeNet and CIFAR-10 quick up to batch 256).
 *   - Allocates no device memory: no hipMalloc / hipFree, no events or
 *     streams, and it never runs the auto-tuner (a conv shape the tuner has
 *     not recorded takes the built-in heuristic).  The scratch is a
 *     file-scope device array, one copy per GPU, held until the process ends;
 *     its device address is looked up once per device on the first call
 *     there.
 *   - x, y, the layer descriptors and the parameters are the caller's, as for
 *     cnn_net_fwd; a network whose cnn_net_workspace_bytes() exceeds
 *     CNN_NOALLOC_SCRATCH_BYTES gets CNN_ERR_WORKSPACE and nothing is
 *     enqueued.
 *   - Every call on one GPU uses the same scratch, which keeps the last pass's
 *     intermediates; a pass writes every intermediate before reading it, so
 *     nothing needs clearing between calls.  Calls that overlap on one GPU
 *     (several streams or threads at once) race on the scratch: the caller
 *     orders them. */
#define CNN_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
int cnn_net_fwd_noalloc(const cnn_layer_desc* layers, int n_layers, const float* x,
                        int N, int C, int H, int W, float* y, cnn_stream_t stream);

/* As cnn_net_fwd, and also writes every layer's output, so that each layer of
 * a network pass can be compared with a reference of that layer (the paper
 * checks only the last layer's output, Sec. 4.1).  A checking aid: the copies
 * cost time and the call is not meant for timing.
 *   dumps    host array of n_layers DEVICE pointers (the array itself must not
 *            be NULL).  dumps[i] NULL: nothing is written for layer i;
 *            otherwise a caller-owned buffer of N*outC*outH*outW floats (the
 *            shape of cnn_net_out_shape over the first i+1 layers) that
 *            receives layer i's output as the layer list defines it: plain
 *            NCHW without the zero border a pooling layer may give its planes
 *            for the padded conv after it, and after the layer's own ReLU even
 *            where the kernel left that ReLU to the next layer's reads.  An
 *            LRN layer run inside the pooling layer after it is run once more
 *            on its own (bit-identical to the fused kernel's LRN values) to
 *            fill its dump.
 *   written  host array of n_layers ints, or NULL: written[i] = 1 where
 *            dumps[i] was filled, 0 where it was NULL or where layer i is a
 *            RELU layer executed inside its predecessor (that predecessor's
 *            dump then holds the output after this ReLU).
 * Validation, errors and the workspace are those of cnn_net_fwd; a dump
 * buffer must not overlap x, y, ws or another dump. */
int cnn_net_fwd_dump(const cnn_layer_desc* layers, int n_layers, const float* x,
                     int N, int C, int H, int W, float* y, void* ws,
                     size_t ws_bytes, float* const* dumps, int* written,
                     cnn_stream_t stream);

/* ---------------------------------------------------------------- execution
 * The paper's engine runs a network either sequentially or in parallel, as
 * the NetFile's execution_mode says (Sec. 3.5).  Here every layer runs on the
 * GPU; the two modes are how the layers reach it: PARALLEL enqueues one
 * network pass per cnn_net_fwd call, GRAPH captures that sequence once into a
 * HIP graph bound to fixed buffers and replays it (one launch per pass).
 */
typedef enum cnn_exec_mode {
    CNN_EXEC_PARALLEL = 0,
    CNN_EXEC_GRAPH = 1
} cnn_exec_mode;

typedef struct cnn_net_graph cnn_net_graph; /* opaque */

/* Captures one cnn_net_fwd(layers, ..., x, y, ws) into a HIP graph; nothing
 * runs.  The graph holds the pointers given here (x, y, ws, the layers'
 * weights, biases and index outputs) and the convolution configurations in
 * force now: a shape that the auto-tuner has not timed yet uses the built-in
 * heuristic, so run the network once with auto-tuning on before capturing to
 * replay tuned configurations.  The layer array itself may be freed after
 * the call.  Returns CNN_OK and *graph, or an error status (validation as in
 * cnn_net_fwd) with *graph = NULL.  Creating a graph allocates host memory and
 * a capture stream; it is not meant for the per-image path. */
int cnn_net_graph_create(const cnn_layer_desc* layers, int n_layers, const float* x,
                         int N, int C, int H, int W, float* y, void* ws,
                         size_t ws_bytes, cnn_net_graph** graph);

/* Enqueues one replay of the graph on `stream` (asynchronous, as cnn_net_fwd). */
int cnn_net_graph_launch(cnn_net_graph* graph, cnn_stream_t stream);

/* Frees the graph (NULL is a no-op).  Replays already enqueued complete. */
int cnn_net_graph_destroy(cnn_net_graph* graph);

/* ---------------------------------------------------------------- NetFile
 * A text description of a network and of the engine's parameters (the
 * paper's NetFile, Sec. 3.2).  One statement per line; '#' starts a comment;
 * "key value" and "key: value" are both accepted for the parameters:
 *   input C H W                     input image shape
 *   execution_mode parallel|graph   (default parallel; "sequential" is
 *                                   CNN_ERR_UNSUPPORTED: no CPU path here)
 *   auto_tuning on|off              (default off)
 *   allocated_ram MIB               parsed and reported only: parameters
 *                                   stay resident in device memory
 * and layer statements, in network order:
 *   conv out=K kernel=R[xS] [stride=..] [pad=..] [groups=G] [in=C] [relu]
 *   fc out=O [in=I] [relu]
 *   pool max|avg kernel=K[xK] [stride=..] [pad=..] [ceil=0|1] [relu]
 *   lrn [size=5] [alpha=1e-4] [beta=0.75] [k=1]
 *   relu
 *   softmax
 * Pairs are "7" or "7x5" (height x width); strides default to 1, pads to 0,
 * ceil to 1 (the pooling rule of cnn_pool_out_shape), groups to 1.  "relu"
 * as an option fuses a ReLU after the layer. */
typedef struct cnn_netfile_config {
    int32_t in_channels, in_height, in_width; /* from "input"; 0 if absent */
    int32_t execution_mode;                    /* cnn_exec_mode */
    int32_t auto_tuning;                       /* 0 or 1 */
    int32_t allocated_ram_mib;                 /* 0 if absent */
} cnn_netfile_config;

/* Parses a NUL-terminated NetFile.  With layers == NULL only counts: sets
 * *n_layers and *config.  Otherwise writes up to max_layers descriptors
 * (weight, bias and pool_index NULL: the caller sets them) and fails with
 * CNN_ERR_INVALID if there are more.  Errors name the line; on error the
 * outputs are unspecified.  Host only, no GPU call. */
int cnn_netfile_parse(const char* text, cnn_layer_desc* layers, int max_layers,
                      int* n_layers, cnn_netfile_config* config);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* cnn_last_error(void);

/* Library version string. */
const char* cnn_version(void);

#ifdef __cplusplus
}
#endif
#endif /* CNN_H */
