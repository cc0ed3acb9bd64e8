// Pooling, local response normalization and ReLU: layers that move far more
// bytes than they compute, so each kernel reads its input once from HBM with
// consecutive lanes on consecutive addresses and writes its output once.
#include "common.h"
#include "fill_jobs.h"

#include <algorithm>
#include <cmath>
#include <vector>

namespace cnn {
namespace {

constexpr int kThreads = 256;

inline int grid_for(int64_t items, int per_thread = 1) {
    const int64_t blocks = (items + (int64_t)kThreads * per_thread - 1) / ((int64_t)kThreads * per_thread);
    return (int)std::max<int64_t>(1, std::min<int64_t>(blocks, 1 << 20));
}

// ------------------------------------------------------------------ pooling
// One thread per output element, lanes along the output row, so the lanes of
// a wave read neighbouring windows of the same input rows.
// v, or max(v, 0) when on: the input of a layer whose producer left its
// ReLU to it (the network executor does so after a split reduction).
__device__ inline float relu_in(float v, int on) { return on ? (v > 0.0f ? v : 0.0f) : v; }

struct PoolParams {
    const float* x;
    float* y;
    int32_t* idx;
    int H, W, P, Q, kh, kw, sh, sw, ph, pw;
    int total;  // N*C*P*Q
    int relu;
    int relu_x;  // take the input through a ReLU as it is read
    int inside;  // no padding and every window lies inside the plane
    FillJobs fills;  // bias fills run after the pooling (n = 0: none)
};

// One pooling window whose KH x KW taps all lie inside the plane (no padding,
// no clipping): t points at its top-left element, ld is the row pitch.  The
// order and the comparisons are those of the clipped loops of the kernels
// below, so the bits are the same: the first maximum in row-major order
// (*rel = its row * ld + column offset from t), or the row-major sum from 0
// (the caller divides by KH * KW, the count of the clipped rule).
template <int MODE, int KH, int KW>
__device__ inline float pool_inside(const float* t, int ld, int* rel) {
    if constexpr (MODE == 0) {
        float best = t[0];
        int bi = 0;
#pragma unroll
        for (int dh = 0; dh < KH; ++dh)
#pragma unroll
            for (int dw = 0; dw < KW; ++dw) {
                if (dh == 0 && dw == 0) continue;
                const float v = t[dh * ld + dw];
                if (v > best) {
                    best = v;
                    bi = dh * ld + dw;
                }
            }
        *rel = bi;
        return best;
    } else {
        float sum = 0.0f;
#pragma unroll
        for (int dh = 0; dh < KH; ++dh)
#pragma unroll
            for (int dw = 0; dw < KW; ++dw) sum += t[dh * ld + dw];
        *rel = 0;
        return sum;
    }
}

template <bool WITH_IDX>
__global__ void __launch_bounds__(kThreads) maxpool_f32(PoolParams p) {
    // 64-bit loop counter: the last step past a total near 2^31 must not wrap
    for (int64_t o64 = blockIdx.x * kThreads + threadIdx.x; o64 < p.total;
         o64 += (int64_t)gridDim.x * kThreads) {
        const int o = (int)o64;
        const int q = o % p.Q;
        const int t = o / p.Q;
        const int pp = t % p.P;
        const int nc = t / p.P;
        const float* plane = p.x + nc * p.H * p.W;
        const int hs = pp * p.sh - p.ph, ws = q * p.sw - p.pw;
        const int h0 = max(hs, 0), w0 = max(ws, 0);
        const int h1 = min(hs + p.kh, p.H), w1 = min(ws + p.kw, p.W);
        // first maximum in row-major order: strict comparison
        int bi = h0 * p.W + w0;
        float best = relu_in(plane[bi], p.relu_x);
        for (int h = h0; h < h1; ++h) {
            const float* row = plane + h * p.W;
            for (int w = w0; w < w1; ++w) {
                const float v = relu_in(row[w], p.relu_x);
                if (v > best) {
                    best = v;
                    bi = h * p.W + w;
                }
            }
        }
        if (p.relu) best = best > 0.0f ? best : 0.0f;
        p.y[o] = best;
        if (WITH_IDX) p.idx[o] = bi;
    }
    run_fills(p.fills);
}


// Pooling with the input staged in LDS: a workgroup takes a run of whole
// (n, c) planes, which is one contiguous stretch of memory, reads it with
// fully coalesced loads into LDS, then computes every output of those planes
// from LDS and writes them contiguously.  Window size and stride are
// template constants for the common 3x3/2 and 2x2/2 windows (KH = 0: taken
// from the parameters).
constexpr int kPoolLdsBytes = 16 * 1024;  // = kThreads * 16 floats: loaded in one round

template <int MODE, bool WITH_IDX, int KH, int KW, int SH, int SW>  // MODE 0: max, 1: average
__global__ void __launch_bounds__(kThreads)
pool_staged_f32(PoolParams p, int planes_per_block, int nplanes, FastDiv fpq, FastDiv fq) {
    extern __shared__ float tile[];
    const int kh = KH ? KH : p.kh, kw = KW ? KW : p.kw;
    const int sh = KH ? SH : p.sh, sw = KW ? SW : p.sw;
    const int HW = p.H * p.W, PQ = p.P * p.Q;
    for (int64_t pl64 = (int64_t)blockIdx.x * planes_per_block; pl64 < nplanes;
         pl64 += (int64_t)gridDim.x * planes_per_block) {
        const int pl0 = (int)pl64;
        const int np = min(planes_per_block, nplanes - pl0);
        const int len = np * HW;
        {  // len <= 16 * kThreads: every load of the run is in flight at once.
           // The buffer resource covers exactly the run, so loads past its end
           // read 0 without a branch.
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<float*>(p.x + (size_t)pl0 * HW), (short)0, len * 4, 0x00020000);
            float v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int i = threadIdx.x + u * kThreads;
                v[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, i * 4, 0, 0));
            }
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int i = threadIdx.x + u * kThreads;
                if (i < len) tile[i] = relu_in(v[u], p.relu_x);
            }
        }
        __syncthreads();
        const int outs = np * PQ;
        if (KH > 0 && p.inside) {  // uniform: windows need no clipping
            for (int o = threadIdx.x; o < outs; o += kThreads) {
                const int pl = (int)fdiv(o, fpq);
                const int r = o - pl * PQ;
                const int pp = (int)fdiv(r, fq);
                const int q = r - pp * p.Q;
                const int corner = pp * sh * p.W + q * sw;
                int rel;
                float out = pool_inside<MODE, KH ? KH : 1, KW ? KW : 1>(tile + pl * HW + corner, p.W, &rel);
                if constexpr (MODE == 1) out = out / (float)(kh * kw);
                if (WITH_IDX && MODE == 0) p.idx[(size_t)pl0 * PQ + o] = corner + rel;
                if (p.relu) out = out > 0.0f ? out : 0.0f;
                p.y[(size_t)pl0 * PQ + o] = out;
            }
            __syncthreads();
            continue;
        }
        for (int o = threadIdx.x; o < outs; o += kThreads) {
            const int pl = (int)fdiv(o, fpq);
            const int r = o - pl * PQ;
            const int pp = (int)fdiv(r, fq);
            const int q = r - pp * p.Q;
            const float* plane = tile + pl * HW;
            const int hs = pp * sh - p.ph, ws = q * sw - p.pw;
            const int h0 = max(hs, 0), w0 = max(ws, 0);
            const int h1 = min(hs + kh, p.H), w1 = min(ws + kw, p.W);
            float out;
            if constexpr (MODE == 0) {
                int bi = h0 * p.W + w0;  // first maximum in row-major order
                float best = plane[bi];
                for (int h = h0; h < h1; ++h)
                    for (int w = w0; w < w1; ++w) {
                        const float v = plane[h * p.W + w];
                        if (v > best) {
                            best = v;
                            bi = h * p.W + w;
                        }
                    }
                out = best;
                if (WITH_IDX) p.idx[(size_t)pl0 * PQ + o] = bi;
            } else {
                const int count = (min(hs + kh, p.H + p.ph) - hs) * (min(ws + kw, p.W + p.pw) - ws);
                float sum = 0.0f;
                for (int h = h0; h < h1; ++h)
                    for (int w = w0; w < w1; ++w) sum += plane[h * p.W + w];
                out = sum / (float)count;
            }
            if (p.relu) out = out > 0.0f ? out : 0.0f;
            p.y[(size_t)pl0 * PQ + o] = out;
        }
        __syncthreads();
    }
    run_fills(p.fills);
}

__global__ void __launch_bounds__(kThreads) avgpool_f32(PoolParams p) {
    for (int64_t o64 = blockIdx.x * kThreads + threadIdx.x; o64 < p.total;
         o64 += (int64_t)gridDim.x * kThreads) {
        const int o = (int)o64;
        const int q = o % p.Q;
        const int t = o / p.Q;
        const int pp = t % p.P;
        const int nc = t / p.P;
        const float* plane = p.x + nc * p.H * p.W;
        const int hs = pp * p.sh - p.ph, ws = q * p.sw - p.pw;
        // divisor: the window clipped to the padded extent
        const int count = (min(hs + p.kh, p.H + p.ph) - hs) * (min(ws + p.kw, p.W + p.pw) - ws);
        const int h0 = max(hs, 0), w0 = max(ws, 0);
        const int h1 = min(hs + p.kh, p.H), w1 = min(ws + p.kw, p.W);
        float sum = 0.0f;
        for (int h = h0; h < h1; ++h) {
            const float* row = plane + h * p.W;
            for (int w = w0; w < w1; ++w) sum += relu_in(row[w], p.relu_x);
        }
        float v = sum / (float)count;
        if (p.relu) v = v > 0.0f ? v : 0.0f;
        p.y[o] = v;
    }
    run_fills(p.fills);
}

// ------------------------------------------------------------------ LRN
// One thread per (n, chunk of CCH channels, pixel); lanes cover consecutive
// pixels.  The thread loads its CCH channels plus a halo of HALF channels on
// each side into registers at once (every load in flight together), then
// forms each channel's window sum from registers.
// Splitting the channels into chunks gives the launch enough threads to keep
// HBM busy even for the 27x27 layers.
struct LrnParams {
    const float* x;
    float* y;
    int C, HW;
    int nchunk;  // ceil(C / CCH)
    int total;   // N * nchunk * H*W
    float alpha_over_size, beta, k;
    int relu_x;  // take the input through a ReLU as it is read
};

// scale^(-beta) through the hardware base-2 logarithm and exponential
// (v_log_f32, v_exp_f32): relative error a few ulp for the scales LRN meets.
__device__ inline float pow_neg(float scale, float beta) {
    return __builtin_amdgcn_exp2f(-beta * __builtin_amdgcn_logf(scale));
}

// One LRN output: w[0 .. WIN-1] are channels c - WIN/2 .. c + WIN/2 at one
// pixel (0 outside the tensor), so w[WIN/2] is x itself.  The standalone and
// the pooling-fused kernels both go through this function, and its roundings
// are spelled out (explicit fused multiply-adds, which the compiler may
// neither split nor share between neighbouring windows), so that the two give
// the same bits.
template <int WIN>
__device__ inline float lrn_value(const float* w, float k, float alpha_over_size, float beta) {
    float sq = w[0] * w[0];
#pragma unroll
    for (int j = 1; j < WIN; ++j) sq = __builtin_fmaf(w[j], w[j], sq);
    return w[WIN / 2] * pow_neg(__builtin_fmaf(alpha_over_size, sq, k), beta);
}

template <int HALF, int CCH>
__global__ void __launch_bounds__(kThreads) lrn_across_f32(LrnParams p) {
    constexpr int WIN = 2 * HALF + 1;
    constexpr int NV = CCH + 2 * HALF;  // channels read per thread
    // Channels outside [0, C) get an out-of-range buffer offset and read 0:
    // the NV loads carry no branch, so all of them are in flight at once.
    const __amdgpu_buffer_rsrc_t xres =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.x), (short)0, 0x7fffffff, 0x00020000);
    for (int64_t t64 = blockIdx.x * kThreads + threadIdx.x; t64 < p.total;
         t64 += (int64_t)gridDim.x * kThreads) {
        const int t = (int)t64;
        const int hw = t % p.HW;
        const int rest = t / p.HW;
        const int chunk = rest % p.nchunk;
        const int n = rest / p.nchunk;
        const int c0 = chunk * CCH;
        const int base = n * p.C * p.HW + hw;  // element (n, 0, hw)
        float v[NV];                            // v[j]: channel c0 - HALF + j
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            const int cc = c0 - HALF + j;
            const int off = (unsigned)cc < (unsigned)p.C ? (base + cc * p.HW) * 4 : (int)0x80000000u;
            v[j] = relu_in(__builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, off, 0, 0)),
                           p.relu_x);
        }
        float* yp = p.y + base;
#pragma unroll
        for (int i = 0; i < CCH; ++i) {  // window of channel c0 + i: v[i] .. v[i + 2 HALF]
            if (c0 + i < p.C) yp[(c0 + i) * p.HW] = lrn_value<WIN>(&v[i], p.k, p.alpha_over_size, p.beta);
        }
    }
}

// LRN followed by pooling in one pass, for the network executor (an LRN layer
// whose output only feeds a pooling layer): the LRN output never goes to
// memory.  A workgroup takes one image, CC channels and a band of PB pooling
// output rows (RB input rows):
//   1. each work-item is one pixel of the band: it loads its CC channels plus
//      the HALF-channel halo on each side straight into registers (every load
//      in flight at once; channels and rows outside the tensor read 0) and
//      writes the CC LRN values to LDS, with the same arithmetic as the LRN
//      kernel;
//   2. pools from the LDS tile (same order and comparisons as the pooling
//      kernels), so the result equals the two layers run one after the other,
//      bit for bit.
// The channel chunk is uniform over the workgroup, so the channel part of
// each load offset is a scalar and a channel outside the tensor is a
// workgroup-wide decision.  Planes (input, LDS band, output) are below 2^24
// elements (checked on the host), so the index arithmetic uses 24-bit
// multiplies.
struct LrnPoolParams {
    const float* x;
    float* y;
    int32_t* idx;
    int C, H, W, P, Q, kh, kw, sh, sw, ph, pw;
    int PB, RB;       // output rows and input rows per workgroup
    int nchunk, nband;
    int relu_x;       // take the input through a ReLU as it is read
    FastDiv f_pbq, f_q;  // PB*OQ, OQ (OQ = Q + 2 opad_w)
    int relu;
    float alpha_over_size, beta, k;
    int opad_h, opad_w;  // y holds each plane inside a zero border of this width
    FillJobs fills;      // bias fills run after the pooling (n = 0: none)
};

__device__ inline int mul24(int a, int b) { return (int)__umul24((unsigned)a, (unsigned)b); }

// KWIN = 3: 3x3 windows of stride 2 that all lie inside the plane (no
// padding), taken with constant offsets; 0: any window, clipped.
template <int HALF, int CC, int MODE, bool WITH_IDX, int KWIN>  // MODE 0: max, 1: average
__global__ void __launch_bounds__(kThreads) lrn_pool_f32(LrnPoolParams p) {
    constexpr int WIN = 2 * HALF + 1;
    constexpr int NV = CC + 2 * HALF;       // channels loaded per work-item
    extern __shared__ float lrn[];          // [CC][RB][W]
    // Workgroups go to the 8 XCDs in turn by id, each XCD with its own L2.
    // Neighbouring channel chunks read the same halo channels, so the ids
    // are remapped to give each XCD a contiguous run of (image, band, chunk)
    // with the chunk fastest: the halo is read from HBM once per XCD run.
    // Ids past the last multiple of 8 keep their position.
    const int nblk = gridDim.x;
    const int full = nblk & ~7;
    const int wg = blockIdx.x;
    int b = wg < full ? (wg & 7) * (full >> 3) + (wg >> 3) : wg;
    const int chunk = b % p.nchunk;
    b /= p.nchunk;
    const int band = b % p.nband;
    const int n = b / p.nband;
    const int c0 = chunk * CC;
    const int p0 = band * p.PB;
    const int pend = min(p0 + p.PB, p.P);
    const int row0 = p0 * p.sh - p.ph;  // first input row of the band (may be < 0)
    const int HW = p.H * p.W;
    const int plane = p.RB * p.W;

    // 1. LRN of the band: work-item `it` is the pixel row0 * W + it of the
    //    image (rows outside the image read 0), channels c0 .. c0 + CC - 1
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(p.x + (size_t)n * p.C * HW), (short)0, 0x7fffffff, 0x00020000);
    const int cs = c0 - HALF;  // channel of v[0]
    const int hw4 = HW * 4;
    for (int it = threadIdx.x; it < plane; it += kThreads) {
        const int pix = row0 * p.W + it;
        const int lane_off = (unsigned)pix < (unsigned)HW ? pix * 4 : (int)0x80000000u;
        // The channel's part of the offset is uniform and goes in the load's
        // scalar offset; for a channel outside the tensor it is 0x7fffffff.
        // The lane's part is at most 2^31 (a pixel offset, or 2^31 for a pixel
        // outside the image), so the sum of the two stays below 2^32, and it
        // reaches the resource's 0x7fffffff bytes, and reads 0, whenever
        // either part is out of range.
        float v[NV];
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            const int c = cs + j;  // uniform
            const int soff = (unsigned)c < (unsigned)p.C ? c * hw4 : 0x7fffffff;
            v[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, lane_off, soff, 0));
        }
        if (p.relu_x) {  // uniform
#pragma unroll
            for (int j = 0; j < NV; ++j) v[j] = relu_in(v[j], 1);
        }
        float* out = lrn + it;
#pragma unroll
        for (int i = 0; i < CC; ++i) out[i * plane] = lrn_value<WIN>(&v[i], p.k, p.alpha_over_size, p.beta);
    }
    __syncthreads();

    // 2. pooling from the LRN tile.  Work-item (c, pr, qq) is column qq of
    //    y's row for output row p0 + pr, border columns included, so that
    //    every row of y is written whole (border columns get 0).
    const int PQ = p.P * p.Q;
    const int OQ = p.Q + 2 * p.opad_w, OPQ = (p.P + 2 * p.opad_h) * OQ;  // y's plane
    const int pbq = p.PB * OQ;
    const int nout = CC * pbq;
    const int nc0 = n * p.C + c0;  // first (image, channel) plane of the workgroup
    float* yw = p.y + (size_t)nc0 * OPQ + (size_t)(p0 + p.opad_h) * OQ;
    for (int o = threadIdx.x; o < nout; o += kThreads) {
        const int c = (int)fdiv(o, p.f_pbq);
        const int rq = o - mul24(c, pbq);
        const int pr = (int)fdiv(rq, p.f_q);
        const int qq = rq - mul24(pr, OQ);
        const int pp = p0 + pr;
        if (c0 + c >= p.C || pp >= pend) continue;
        const int q = qq - p.opad_w;
        float out = 0.0f;
        if (KWIN == 3 && (unsigned)q < (unsigned)p.Q) {
            const int hs = pp * 2, ws = q * 2;
            int rel;
            out = pool_inside<MODE, 3, 3>(lrn + mul24(c, plane) + mul24(hs - row0, p.W) + ws, p.W, &rel);
            if constexpr (MODE == 1) out = out / 9.0f;
            if (WITH_IDX && MODE == 0)
                p.idx[(size_t)(nc0 + c) * PQ + mul24(pp, p.Q) + q] = mul24(hs, p.W) + ws + rel;
            if (p.relu) out = out > 0.0f ? out : 0.0f;
        } else if ((unsigned)q < (unsigned)p.Q) {
            const int hs = pp * p.sh - p.ph, ws = q * p.sw - p.pw;
            const int h0 = max(hs, 0), w0 = max(ws, 0);
            const int h1 = min(hs + p.kh, p.H), w1 = min(ws + p.kw, p.W);
            const float* t = lrn + mul24(c, plane);
            if constexpr (MODE == 0) {
                int bi = h0 * p.W + w0;  // first maximum in row-major order
                float best = t[(h0 - row0) * p.W + w0];
                for (int h = h0; h < h1; ++h)
                    for (int w = w0; w < w1; ++w) {
                        const float v = t[(h - row0) * p.W + w];
                        if (v > best) {
                            best = v;
                            bi = h * p.W + w;
                        }
                    }
                out = best;
                if (WITH_IDX) p.idx[(size_t)(nc0 + c) * PQ + pp * p.Q + q] = bi;
            } else {
                const int count = (min(hs + p.kh, p.H + p.ph) - hs) * (min(ws + p.kw, p.W + p.pw) - ws);
                float sum = 0.0f;
                for (int h = h0; h < h1; ++h)
                    for (int w = w0; w < w1; ++w) sum += t[(h - row0) * p.W + w];
                out = sum / (float)count;
            }
            if (p.relu) out = out > 0.0f ? out : 0.0f;
        }
        yw[mul24(c, OPQ) + rq] = out;
    }

    // 3. y's border rows above the first band and below the last, whole rows
    if (p.opad_h > 0 && (p0 == 0 || pend == p.P)) {
        const int per_c = p.opad_h * OQ;  // border elements above (or below) a plane
        const int nedge = (p0 == 0) + (pend == p.P);
        for (int o = threadIdx.x; o < CC * nedge * per_c; o += kThreads) {
            const int ce = o / per_c;  // (channel, edge)
            const int e = o - ce * per_c;
            const int c = ce / nedge;
            const bool below = (ce - c * nedge) == 1 || p0 != 0;
            const int off = below ? (p.opad_h + p.P) * OQ + e : e;
            if (c0 + c < p.C) p.y[(size_t)(nc0 + c) * OPQ + off] = 0.0f;
        }
    }
    run_fills(p.fills);
}

// Any odd size: recompute the clipped window sum for every channel.
__global__ void __launch_bounds__(kThreads) lrn_across_any_f32(LrnParams p, int half) {
    for (int64_t t64 = blockIdx.x * kThreads + threadIdx.x; t64 < p.total;
         t64 += (int64_t)gridDim.x * kThreads) {
        const int t = (int)t64;
        const int n = t / p.HW;
        const int hw = t - n * p.HW;
        const float* xp = p.x + n * p.C * p.HW + hw;
        float* yp = p.y + n * p.C * p.HW + hw;
        for (int c = 0; c < p.C; ++c) {
            const int c0 = max(c - half, 0), c1 = min(c + half, p.C - 1);
            float sq = 0.0f;
            for (int cc = c0; cc <= c1; ++cc) {
                const float v = relu_in(xp[cc * p.HW], p.relu_x);
                sq += v * v;
            }
            const float scale = p.k + p.alpha_over_size * sq;
            yp[c * p.HW] = relu_in(xp[c * p.HW], p.relu_x) * pow_neg(scale, p.beta);
        }
    }
}

// ------------------------------------------------------------------ ReLU
__device__ inline float relu1(float v) { return v > 0.0f ? v : 0.0f; }

__global__ void __launch_bounds__(kThreads) relu_f32x4(const float4* x, float4* y, int64_t n4) {
    for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < n4;
         i += (int64_t)gridDim.x * kThreads) {
        const float4 v = x[i];
        y[i] = make_float4(relu1(v.x), relu1(v.y), relu1(v.z), relu1(v.w));
    }
}

__global__ void __launch_bounds__(kThreads) relu_f32(const float* x, float* y, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads)
        y[i] = relu1(x[i]);
}

// ------------------------------------------------------------------ copies
// dst[plane][p][q] = src[plane][p + bh][q + bw] (source planes of
// (P + 2 bh) x (Q + 2 bw)), through a ReLU when `relu` is set: the layer
// outputs a network pass writes out for checking.
__global__ void __launch_bounds__(kThreads) copy_planes_f32(const float* src, float* dst, int64_t total,
                                                            int P, int Q, int bh, int bw, int relu) {
    const int64_t PQ = (int64_t)P * Q, QB = Q + 2 * bw, PQB = (int64_t)(P + 2 * bh) * QB;
    for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * kThreads) {
        const int64_t plane = i / PQ, r = i - plane * PQ;
        const int64_t p = r / Q, q = r - p * Q;
        const float v = src[plane * PQB + (p + bh) * QB + q + bw];
        dst[i] = relu ? relu1(v) : v;
    }
}

}  // namespace

int launch_copy_planes(const float* src, float* dst, int64_t planes, int P, int Q, int bh, int bw,
                       bool relu, hipStream_t st) {
    const int64_t total = planes * P * Q;
    if (total == 0) return CNN_OK;
    enqueue(copy_planes_f32, dim3(grid_for(total)), dim3(kThreads), 0, st, src, dst, total, P, Q,
                       bh, bw, (int)relu);
    return check_launch("copy_planes_f32");
}

int launch_pool(const PoolShape& s, int mode, int relu, const float* x, float* y, int32_t* idx,
                hipStream_t st, bool relu_x, const FillJobs* fills) {
    PoolParams p;
    p.relu_x = relu_x;
    p.fills.n = 0;
    if (fills) p.fills = *fills;
    p.x = x;
    p.y = y;
    p.idx = idx;
    p.H = s.H; p.W = s.W; p.P = s.P; p.Q = s.Q;
    p.kh = s.kh; p.kw = s.kw; p.sh = s.sh; p.sw = s.sw; p.ph = s.ph; p.pw = s.pw;
    p.total = s.N * s.C * s.P * s.Q;
    p.relu = relu;
    p.inside = s.ph == 0 && s.pw == 0 && (int64_t)(s.P - 1) * s.sh + s.kh <= s.H &&
               (int64_t)(s.Q - 1) * s.sw + s.kw <= s.W;
    if (p.total == 0) return fills ? launch_bias_fills(fills->job, fills->n, st) : CNN_OK;
    const int plane_bytes = s.H * s.W * 4;
    if (plane_bytes <= kPoolLdsBytes) {
        // planes per workgroup: as many as the staging buffer holds, but no
        // more than leaves ~2048 workgroups, so that small layers still
        // spread over every CU
        const int nplanes = s.N * s.C;
        const int ppb = std::max(1, std::min(kPoolLdsBytes / plane_bytes, nplanes / 2048));
        const dim3 g(std::min(ceil_div(nplanes, ppb), 1 << 20)), b(kThreads);
        const size_t shm = (size_t)ppb * plane_bytes;
        const FastDiv fpq = make_fastdiv(s.P * s.Q), fq = make_fastdiv(s.Q);
        const bool w33 = s.kh == 3 && s.kw == 3 && s.sh == 2 && s.sw == 2;
        const bool w22 = s.kh == 2 && s.kw == 2 && s.sh == 2 && s.sw == 2;
#define CNN_POOL_LAUNCH(M, I)                                                                              \
    do {                                                                                                   \
        if (w33)                                                                                           \
            enqueue((pool_staged_f32<M, I, 3, 3, 2, 2>), g, b, shm, st, p, ppb, nplanes, fpq, fq); \
        else if (w22)                                                                                      \
            enqueue((pool_staged_f32<M, I, 2, 2, 2, 2>), g, b, shm, st, p, ppb, nplanes, fpq, fq); \
        else                                                                                               \
            enqueue((pool_staged_f32<M, I, 0, 0, 0, 0>), g, b, shm, st, p, ppb, nplanes, fpq, fq); \
    } while (0)
        if (mode == CNN_POOL_MAX && idx)
            CNN_POOL_LAUNCH(0, true);
        else if (mode == CNN_POOL_MAX)
            CNN_POOL_LAUNCH(0, false);
        else
            CNN_POOL_LAUNCH(1, false);
#undef CNN_POOL_LAUNCH
        return check_launch("pool_staged_f32");
    }
    // planes larger than the staging buffer: one thread per output from memory
    const dim3 grid(grid_for(p.total)), block(kThreads);
    if (mode == CNN_POOL_MAX) {
        if (idx)
            enqueue(maxpool_f32<true>, grid, block, 0, st, p);
        else
            enqueue(maxpool_f32<false>, grid, block, 0, st, p);
        return check_launch("maxpool_f32");
    }
    enqueue(avgpool_f32, grid, block, 0, st, p);
    return check_launch("avgpool_f32");
}

int launch_lrn(const float* x, int N, int C, int H, int W, int size, float alpha, float beta,
               float k, float* y, hipStream_t st, bool relu_x) {
    LrnParams p;
    p.relu_x = relu_x;
    p.x = x;
    p.y = y;
    p.C = C;
    p.HW = H * W;
    p.alpha_over_size = alpha / (float)size;
    p.beta = beta;
    p.k = k;
    if (N == 0) return CNN_OK;
    constexpr int kChunk = 32;
    const int64_t img = (int64_t)C * p.HW;
    if (size / 2 > 4 || img >= ((int64_t)1 << 29)) {  // wide windows, huge images
        p.nchunk = 1;
        p.total = N * p.HW;
        enqueue(lrn_across_any_f32, dim3(grid_for(p.total)), dim3(kThreads), 0, st, p,
                           size / 2);
        return check_launch("lrn_across_any_f32");
    }
    // The chunked kernel addresses x through a buffer resource with 31-bit
    // byte offsets: fewer than 2^29 elements per launch (whole images).
    const int per_launch = (int)std::min<int64_t>(N, (((int64_t)1 << 29) - 1) / img);
    p.nchunk = ceil_div(C, kChunk);
    for (int n0 = 0; n0 < N; n0 += per_launch) {
        const int nb = std::min(per_launch, N - n0);
        p.x = x + (size_t)n0 * img;
        p.y = y + (size_t)n0 * img;
        p.total = nb * p.nchunk * p.HW;
        const dim3 grid(grid_for(p.total)), block(kThreads);
        switch (size / 2) {
            case 0: enqueue((lrn_across_f32<0, kChunk>), grid, block, 0, st, p); break;
            case 1: enqueue((lrn_across_f32<1, kChunk>), grid, block, 0, st, p); break;
            case 2: enqueue((lrn_across_f32<2, kChunk>), grid, block, 0, st, p); break;
            case 3: enqueue((lrn_across_f32<3, kChunk>), grid, block, 0, st, p); break;
            default: enqueue((lrn_across_f32<4, kChunk>), grid, block, 0, st, p); break;
        }
        const int rc = check_launch("lrn_across_f32");
        if (rc != CNN_OK) return rc;
    }
    return CNN_OK;
}

namespace {
struct LrnPoolTiling {
    int CB, CC, PB, RB;
    int64_t blocks;
};

// Channels (CB, with CC = CB per work-item) and output rows per workgroup of
// the fused LRN + pooling kernel.  The kernel is bound by how many loads are
// in flight, so occupancy comes first: a workgroup keeps its LDS tile within
// 20 KB, which lets 8 workgroups (32 waves) share a CU; only shapes with no
// such tiling go up to 40 KB.  Among those tilings the cheapest reads the
// fewest input elements per LRN value it keeps (channel halo times
// overlapping band rows), with ragged passes of the workgroup over its
// work-items counted in full.  A launch needs enough workgroups to fill the
// chip: tilings giving fewer than 1024 (or than the most any tiling gives,
// for small batches) are passed over.  False when nothing fits.
bool lrn_pool_tiling(const PoolShape& s, int half, LrnPoolTiling* t) {
    for (int budget : {20 * 1024, 40 * 1024}) {
        std::vector<LrnPoolTiling> cand;
        std::vector<double> cost;
        int64_t most = 0;
        for (int cb : {16, 8}) {
            if (cb > 8 && cb / 2 >= s.C) continue;  // no wider than the channels need
            for (int pb = 1; pb <= std::min(s.P, 16); ++pb) {
                const int rb = (pb - 1) * s.sh + s.kh;
                if ((int64_t)cb * rb * s.W * 4 > budget) break;
                const int64_t items = (int64_t)rb * s.W;
                const double fill = (double)ceil_div64(items, kThreads) * kThreads / (double)items;
                const double amp = (double)(cb + 2 * half) / std::min(cb, s.C) * rb / ((double)pb * s.sh);
                cand.push_back({cb, cb, pb, rb, (int64_t)s.N * ceil_div(s.C, cb) * ceil_div(s.P, pb)});
                cost.push_back(amp * fill);
                most = std::max(most, cand.back().blocks);
            }
        }
        const int64_t want = std::min<int64_t>(1024, most);
        double best = 1e30;
        for (size_t i = 0; i < cand.size(); ++i)
            if (cand[i].blocks >= want && cost[i] < best - 1e-12) {
                best = cost[i];
                *t = cand[i];
            }
        if (best < 1e29) return true;
    }
    return false;
}
}  // namespace

bool lrn_pool_fusable(const PoolShape& s, int size) {
    LrnPoolTiling t;
    // the kernel's 24-bit index products: input and output planes below
    // 2^24 elements (a bordered output plane is checked by the caller)
    if (size % 2 != 1 || size / 2 > 4 || (int64_t)s.C * s.H * s.W >= ((int64_t)1 << 29) ||
        (int64_t)s.H * s.W >= ((int64_t)1 << 24) || !lrn_pool_tiling(s, size / 2, &t))
        return false;
    return t.blocks * kThreads < ((int64_t)1 << 32);  // the launch's work-items fit 32 bits
}

int launch_lrn_pool(const PoolShape& s, int mode, int relu, int size, float alpha, float beta, float k,
                    const float* x, float* y, int32_t* idx, hipStream_t st, bool relu_x,
                    const FillJobs* fills, int opad_h, int opad_w) {
    if (s.N == 0) return fills ? launch_bias_fills(fills->job, fills->n, st) : CNN_OK;
    const int half = size / 2;
    LrnPoolTiling t;
    if (!lrn_pool_fusable(s, size) || !lrn_pool_tiling(s, half, &t))
        return fail(CNN_ERR_UNSUPPORTED, "lrn+pool: no fused tiling for this shape");
    const int64_t ohb = (int64_t)s.P + 2 * (int64_t)opad_h, owb = (int64_t)s.Q + 2 * (int64_t)opad_w;
    if (opad_h < 0 || opad_w < 0 || ohb >= ((int64_t)1 << 24) || owb >= ((int64_t)1 << 24) ||
        ohb * owb >= ((int64_t)1 << 24))
        return fail(CNN_ERR_UNSUPPORTED, "lrn+pool: bordered output plane of 2^24 elements or more");
    LrnPoolParams p;
    p.x = x;
    p.y = y;
    p.idx = idx;
    p.C = s.C; p.H = s.H; p.W = s.W; p.P = s.P; p.Q = s.Q;
    p.kh = s.kh; p.kw = s.kw; p.sh = s.sh; p.sw = s.sw; p.ph = s.ph; p.pw = s.pw;
    p.PB = t.PB;
    p.RB = t.RB;
    p.nchunk = ceil_div(s.C, t.CB);
    p.nband = ceil_div(s.P, p.PB);
    p.f_pbq = make_fastdiv(p.PB * (s.Q + 2 * opad_w));  // y's rows hold the border columns too
    p.f_q = make_fastdiv(s.Q + 2 * opad_w);
    p.relu = relu;
    p.alpha_over_size = alpha / (float)size;
    p.beta = beta;
    p.k = k;
    p.relu_x = relu_x;
    p.opad_h = opad_h;
    p.opad_w = opad_w;
    p.fills.n = 0;
    if (fills) p.fills = *fills;
    const size_t shm = (size_t)t.CB * p.RB * s.W * 4;
    const dim3 grid((unsigned)t.blocks), block(kThreads);
    // 3x3 windows of stride 2 inside the plane (AlexNet's pooling) take the
    // constant-offset window for the five-channel LRN
    const bool win3 = half == 2 && s.kh == 3 && s.kw == 3 && s.sh == 2 && s.sw == 2 && s.ph == 0 &&
                      s.pw == 0 && (s.P - 1) * 2 + 3 <= s.H && (s.Q - 1) * 2 + 3 <= s.W;
#define CNN_LRN_POOL_CC(H, CC, KW)                                                                   \
    do {                                                                                             \
        if (mode == CNN_POOL_MAX && idx)                                                             \
            enqueue((lrn_pool_f32<H, CC, 0, true, KW>), grid, block, shm, st, p);         \
        else if (mode == CNN_POOL_MAX)                                                               \
            enqueue((lrn_pool_f32<H, CC, 0, false, KW>), grid, block, shm, st, p);        \
        else                                                                                         \
            enqueue((lrn_pool_f32<H, CC, 1, false, KW>), grid, block, shm, st, p);        \
    } while (0)
#define CNN_LRN_POOL(H, KW)                  \
    do {                                     \
        if (t.CC == 16)                      \
            CNN_LRN_POOL_CC(H, 16, KW);      \
        else                                 \
            CNN_LRN_POOL_CC(H, 8, KW);       \
    } while (0)
    switch (half) {
        case 0: CNN_LRN_POOL(0, 0); break;
        case 1: CNN_LRN_POOL(1, 0); break;
        case 2:
            if (win3)
                CNN_LRN_POOL(2, 3);
            else
                CNN_LRN_POOL(2, 0);
            break;
        case 3: CNN_LRN_POOL(3, 0); break;
        default: CNN_LRN_POOL(4, 0); break;
    }
#undef CNN_LRN_POOL
#undef CNN_LRN_POOL_CC
    return check_launch("lrn_pool_f32");
}

int launch_relu(const float* x, float* y, int64_t n, hipStream_t st) {
    if (n == 0) return CNN_OK;
    const bool vec = ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y)) & 15) == 0;
    int64_t done = 0;
    if (vec && n >= 4) {
        const int64_t n4 = n / 4;
        enqueue(relu_f32x4, dim3(grid_for(n4, 4)), dim3(kThreads), 0, st,
                           reinterpret_cast<const float4*>(x), reinterpret_cast<float4*>(y), n4);
        done = n4 * 4;
    }
    if (done < n)
        enqueue(relu_f32, dim3(grid_for(n - done)), dim3(kThreads), 0, st, x + done,
                           y + done, n - done);
    return check_launch("relu_f32");
}

}  // namespace cnn
