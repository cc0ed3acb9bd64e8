// Convolution layer as an implicit GEMM on the fp32 matrix cores of gfx950.
//
// Per group g the layer is the product
//     Y_g[k][m] = sum_kk W_g[k][kk] * X_g[kk][m]      (+ bias, optional ReLU)
// with k an output channel of the group (Kg = K/G rows), m = (n, p, q) an
// output pixel (M = N*P*Q columns) and kk = (c, r, s) a tap of the filter
// (Kr = (C/G)*R*S, in the weights' own [c][r][s] order).  X_g is the im2col
// matrix of the input; it is never built in memory: each workgroup gathers the
// slab of it that it needs straight from the NCHW input into LDS.
//
// Gather: every thread owns one output pixel (fixed for the whole kernel) and
// a run of consecutive taps per slab; the taps' (c, r, s) are wave-uniform and
// advance in scalar registers.  Loads go through a buffer resource: a tap
// that falls into the zero padding, or past the end of the reduction, gets an
// out-of-range offset and the hardware returns 0, so the gather has no
// branches.
//
// Workgroup tile: TM output channels x TN output pixels, reduction in slabs of
// BK taps, double-buffered in LDS (the loads of slab s+1 are in flight while
// slab s feeds the matrix cores).  Each wave owns FM x FN blocks of 32x32
// accumulated with v_mfma_f32_32x32x2_f32.  The output channel is the MFMA
// row and the output pixel the MFMA column, so the 32 lanes of a row store 32
// consecutive pixels: NCHW stores are coalesced.
//
// Reduction order inside a slab: lanes 0-31 take the first BK/2 taps of the
// slab and lanes 32-63 the last BK/2 (an MFMA step consumes one tap per lane
// half), so each lane reads BK/2 consecutive LDS words per fragment with
// 128-bit loads.  The order of a sum changes its value only by rounding.
#include <cstdlib>
#include <cstring>

#include "common.h"

namespace cnn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kOutOfRange = (int)0x80000000u;  // buffer offset that reads as 0

struct ConvParams {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int C, H, W, K, R, S, P, Q;
    int sh, sw, ph, pw;
    int Cg, Kg, Kr, RS, HW, PQ, M;
    int xbytes;  // bytes of x covered by this launch (< 2^31)
    int relu;
};

template <int WMW, int WNW, int FM, int FN, int BK, bool VEC_W>
__global__ void __launch_bounds__(64 * WMW * WNW)
conv2d_igemm_f32(ConvParams p) {
    constexpr int TM = WMW * FM * 32;  // output channels per workgroup
    constexpr int TN = WNW * FN * 32;  // output pixels per workgroup
    constexpr int NT = 64 * WMW * WNW;
    constexpr int LDK = BK + 4;        // padded LDS row (conflict-free 128-bit reads)
    constexpr int KGROUPS = NT / TN;   // threads sharing one pixel column of the gather
    constexpr int KRUN = BK / KGROUPS; // consecutive taps gathered per thread
    static_assert(NT % TN == 0 && TN >= 64, "gather layout needs TN | NT and TN >= 64");
    static_assert(BK % KGROUPS == 0 && KRUN % 4 == 0, "gather run must be whole float4s");
    static_assert(BK % 8 == 0, "slab must split into two halves of float4s");
    constexpr int WTOT = VEC_W ? TM * BK / 4 : TM * BK;  // weight-tile loads per slab
    constexpr int WV = (WTOT + NT - 1) / NT;                // ... per thread (last one guarded)

    __shared__ __attribute__((aligned(16))) float sA[2][TM * LDK];  // weights  [k][kk]
    __shared__ __attribute__((aligned(16))) float sB[2][TN * LDK];  // im2col   [m][kk]

    const int tid = threadIdx.x;
    const int g = blockIdx.z;
    const int m0 = blockIdx.x * TN;
    const int k0 = blockIdx.y * TM;

    // ---- gather setup: this thread's pixel and tap run (fixed for all slabs)
    const int mloc = tid % TN;
    const int kgrp = __builtin_amdgcn_readfirstlane(tid / TN);  // uniform: TN >= 64
    const int m = m0 + mloc;
    int hb, wb, lane_off;
    if (m < p.M) {
        const int n = m / p.PQ;
        const int pq = m - n * p.PQ;
        const int pp = pq / p.Q;
        const int qq = pq - pp * p.Q;
        hb = pp * p.sh - p.ph;
        wb = qq * p.sw - p.pw;
        lane_off = ((n * p.C + g * p.Cg) * p.HW + hb * p.W + wb) * 4;
    } else {
        hb = -0x40000000;  // every row test fails: the column reads as zero
        wb = 0;
        lane_off = 0;
    }
    const __amdgpu_buffer_rsrc_t xres =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.x), (short)0, p.xbytes, 0x00020000);

    float xr[KRUN];
    auto load_x = [&](int kslab) {
        const int kk0 = kslab + kgrp * KRUN;  // uniform
        int c = kk0 / p.RS;
        const int rs = kk0 - c * p.RS;
        int r = rs / p.S;
        int s = rs - r * p.S;
        int toff = ((c * p.H + r) * p.W + s) * 4;  // byte offset of tap (c, r, s)
#pragma unroll
        for (int j = 0; j < KRUN; ++j) {
            const bool ok = (kk0 + j < p.Kr) && ((unsigned)(hb + r) < (unsigned)p.H) &&
                            ((unsigned)(wb + s) < (unsigned)p.W);
            const int voff = ok ? lane_off + toff : kOutOfRange;
            xr[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, voff, 0, 0));
            // next tap: s, then r, then c
            ++s;
            toff += 4;
            const bool wrap_s = (s == p.S);
            s = wrap_s ? 0 : s;
            r += wrap_s ? 1 : 0;
            toff += wrap_s ? (p.W - p.S) * 4 : 0;
            const bool wrap_r = (r == p.R);
            r = wrap_r ? 0 : r;
            toff += wrap_r ? (p.HW - p.R * p.W) * 4 : 0;
        }
    };
    auto store_x = [&](int buf) {
        float* dst = &sB[buf][mloc * LDK + kgrp * KRUN];
#pragma unroll
        for (int j = 0; j < KRUN; j += 4)
            *reinterpret_cast<float4*>(dst + j) = make_float4(xr[j], xr[j + 1], xr[j + 2], xr[j + 3]);
    };

    // ---- weight tile loads: rows k0.. of the group's [Kg][Kr] block
    const float* wg = p.w + g * p.Kg * p.Kr;
    float4 wr4[VEC_W ? WV : 1];
    float wr1[VEC_W ? 1 : WV];
    auto load_w = [&](int kslab) {
#pragma unroll
        for (int i = 0; i < WV; ++i) {
            const int idx = tid + i * NT;
            if (WTOT % NT != 0 && idx >= WTOT) break;
            if constexpr (VEC_W) {
                const int row = idx / (BK / 4);
                const int col = (idx % (BK / 4)) * 4;
                const int kr = k0 + row, kk = kslab + col;
                wr4[i] = (kr < p.Kg && kk < p.Kr)
                             ? *reinterpret_cast<const float4*>(wg + kr * p.Kr + kk)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
            } else {
                const int row = idx / BK;
                const int col = idx % BK;
                const int kr = k0 + row, kk = kslab + col;
                wr1[i] = (kr < p.Kg && kk < p.Kr) ? wg[kr * p.Kr + kk] : 0.0f;
            }
        }
    };
    auto store_w = [&](int buf) {
#pragma unroll
        for (int i = 0; i < WV; ++i) {
            const int idx = tid + i * NT;
            if (WTOT % NT != 0 && idx >= WTOT) break;
            if constexpr (VEC_W) {
                const int row = idx / (BK / 4);
                const int col = (idx % (BK / 4)) * 4;
                *reinterpret_cast<float4*>(&sA[buf][row * LDK + col]) = wr4[i];
            } else {
                const int row = idx / BK;
                const int col = idx % BK;
                sA[buf][row * LDK + col] = wr1[i];
            }
        }
    };

    // ---- matrix-core work of one slab
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WNW;
    const int wn = wave % WNW;
    const int half = lane >> 5;
    const int l32 = lane & 31;
    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    auto compute = [&](int buf) {
        float a[FM][BK / 2];
        float b[FN][BK / 2];
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const float* src = &sA[buf][(wm * FM * 32 + i * 32 + l32) * LDK + half * (BK / 2)];
#pragma unroll
            for (int t = 0; t < BK / 2; t += 4) {
                const float4 v = *reinterpret_cast<const float4*>(src + t);
                a[i][t] = v.x; a[i][t + 1] = v.y; a[i][t + 2] = v.z; a[i][t + 3] = v.w;
            }
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const float* src = &sB[buf][(wn * FN * 32 + j * 32 + l32) * LDK + half * (BK / 2)];
#pragma unroll
            for (int t = 0; t < BK / 2; t += 4) {
                const float4 v = *reinterpret_cast<const float4*>(src + t);
                b[j][t] = v.x; b[j][t + 1] = v.y; b[j][t + 2] = v.z; b[j][t + 3] = v.w;
            }
        }
#pragma unroll
        for (int t = 0; t < BK / 2; ++t)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][t], b[j][t], acc[i][j], 0, 0, 0);
    };

    // ---- main loop: slab s computes from LDS while slab s+1 loads from memory
    const int nslab = (p.Kr + BK - 1) / BK;
    load_x(0);
    load_w(0);
    store_x(0);
    store_w(0);
    __syncthreads();
    for (int sl = 0; sl < nslab; ++sl) {
        const int cur = sl & 1;
        const bool more = sl + 1 < nslab;
        if (more) {
            load_x((sl + 1) * BK);
            load_w((sl + 1) * BK);
        }
        compute(cur);
        if (more) {
            store_x(cur ^ 1);
            store_w(cur ^ 1);
        }
        __syncthreads();
    }

    // ---- epilogue: bias, ReLU, NCHW store (lanes = consecutive pixels)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int mc = m0 + wn * FN * 32 + j * 32 + l32;
        if (mc >= p.M) continue;
        const int n = mc / p.PQ;
        const int pq = mc - n * p.PQ;
        float* yb = p.y + n * p.K * p.PQ + pq;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int kr = k0 + wm * FM * 32 + i * 32 + 8 * (v / 4) + 4 * half + (v % 4);
                if (kr < p.Kg) {
                    const int ko = g * p.Kg + kr;
                    float val = acc[i][j][v];
                    if (p.bias) val += p.bias[ko];
                    if (p.relu) val = val > 0.0f ? val : 0.0f;
                    yb[ko * p.PQ] = val;
                }
            }
        }
    }
}

// ---------------------------------------------------------------- configurations
typedef int (*LaunchFn)(const ConvParams&, int G, bool vec_w, hipStream_t st);

template <int WMW, int WNW, int FM, int FN, int BK>
int launch_cfg(const ConvParams& prm, int G, bool vec_w, hipStream_t st) {
    constexpr int TM = WMW * FM * 32;
    constexpr int TN = WNW * FN * 32;
    dim3 grid(ceil_div(prm.M, TN), ceil_div(prm.Kg, TM), G);
    dim3 block(64 * WMW * WNW);
    if (vec_w)
        hipLaunchKernelGGL((conv2d_igemm_f32<WMW, WNW, FM, FN, BK, true>), grid, block, 0, st, prm);
    else
        hipLaunchKernelGGL((conv2d_igemm_f32<WMW, WNW, FM, FN, BK, false>), grid, block, 0, st, prm);
    return check_launch("conv2d_igemm_f32");
}

struct ConvConfig {
    const char* name;  // "TMxTNxBK"
    int tm, tn, bk, threads;
    LaunchFn launch;
};

#define CNN_CONV_CFG(WMW, WNW, FM, FN, BK)                                                       \
    ConvConfig {                                                                                \
        #WMW "x" #WNW " waves, " #FM "x" #FN " blocks, BK " #BK, WMW * FM * 32, WNW * FN * 32, \
            BK, 64 * WMW * WNW, &launch_cfg<WMW, WNW, FM, FN, BK>                               \
    }

const ConvConfig kConfigs[] = {
    CNN_CONV_CFG(2, 2, 2, 2, 16),  // 0: 128 x 128
    CNN_CONV_CFG(2, 2, 2, 2, 32),  // 1: 128 x 128
    CNN_CONV_CFG(4, 1, 1, 2, 16),  // 2: 128 x 64
    CNN_CONV_CFG(4, 1, 1, 2, 32),  // 3: 128 x 64
    CNN_CONV_CFG(1, 4, 2, 1, 16),  // 4: 64 x 128
    CNN_CONV_CFG(1, 4, 2, 1, 32),  // 5: 64 x 128
    CNN_CONV_CFG(1, 4, 3, 1, 16),  // 6: 96 x 128
    CNN_CONV_CFG(1, 4, 3, 1, 32),  // 7: 96 x 128
    CNN_CONV_CFG(1, 4, 1, 1, 16),  // 8: 32 x 128
    CNN_CONV_CFG(2, 2, 1, 1, 16),  // 9: 64 x 64
    CNN_CONV_CFG(2, 2, 1, 1, 32),  // 10: 64 x 64
    CNN_CONV_CFG(2, 4, 2, 2, 16),  // 11: 128 x 256 (8 waves)
    CNN_CONV_CFG(1, 2, 3, 2, 16),  // 12: 96 x 128 (2 waves)
    CNN_CONV_CFG(2, 1, 2, 2, 16),  // 13: 128 x 64 (2 waves)
};
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
