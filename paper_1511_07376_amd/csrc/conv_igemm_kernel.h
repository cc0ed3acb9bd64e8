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
// a run of consecutive taps per slab, whose (c, r, s) are wave-uniform: read
// from a per-workgroup tap table in LDS for filters of at most 31 taps, else
// advanced in scalar registers.  Loads go through a buffer resource: a tap
// that falls into the zero padding, or past the end of the reduction, gets an
// out-of-range offset and the hardware returns 0, so the gather has no
// branches.
//
// Workgroup tile: TM output channels x TN output pixels, reduction in slabs of
// BK taps, double-buffered in LDS, with the loads of the next ST slabs in
// flight in ST register stages while slab s feeds the matrix cores.  Each
// wave owns FM x FN blocks of 32x32 accumulated with v_mfma_f32_32x32x2_f32.
// The output channel is the MFMA row and the output pixel the MFMA column,
// so the 32 lanes of a row store 32 consecutive pixels: NCHW stores are
// coalesced.
//
// Reduction order inside a slab: lanes 0-31 take the first BK/2 taps of the
// slab and lanes 32-63 the last BK/2 (an MFMA step consumes one tap per lane
// half), so each lane reads BK/2 consecutive LDS words per fragment with
// 128-bit loads.  The order of a sum changes its value only by rounding.
//
// Split reduction: when the output has too few tiles to occupy the chip (a
// batch of one image, say), grid z also splits the reduction into chunks of
// kchunk taps; each workgroup then adds its partial tile into an output that
// holds the bias already, with fp32 atomics, and a ReLU, if any, runs after
// the last chunk.
#pragma once

#include <cstdlib>
#include <cstring>

#include "common.h"

namespace cnn {
namespace conv {

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
    int wbytes;  // bytes of w (< 2^31)
    int relu;
    int relu_x;  // take the input through a ReLU as it is gathered
    int G;       // groups (grid z = G * splits)
    int splits;  // reduction chunks; > 1: partial tiles are added atomically
    int kchunk;  // taps per chunk (a multiple of every slab length; Kr if splits == 1)
    FastDiv f_rs, f_s, f_pq, f_q;  // division by R*S, S, P*Q and Q
};

// Gather modes.
//  kGatherScalar: taps decoded and advanced in scalar registers, bounds
//    tested per element (any filter).
//  kGatherMask: filters of at most 31 taps.  A tap table in LDS, built once
//    per workgroup, holds entry kk = (byte offset of tap kk within an image
//    group) << 5 | (r*S + s); tap index 31 marks "past the reduction".  Each
//    thread builds once a 32-bit mask of the (r, s) taps that fall outside
//    the image for its pixel (bit 31 always set).  An element costs a mask
//    bit test, an add and an OR of the out-of-range bit into the offset.
//  kGatherNoPad: no padding, so every tap of an in-range pixel lies inside
//    the image.  The table holds byte offsets (2^31 past the reduction) and
//    out-of-range pixels start at 2^31: an element costs one add.
//  kGatherStrided: no padding and a column stride above 1.  Same table, but
//    one load instruction covers 16 neighbouring pixels x 4 consecutive taps
//    (lane l: pixel l/4, tap l%4) instead of 64 pixels x 1 tap: with
//    neighbouring pixels `stride` floats apart, the 64 addresses then span 2-3
//    cache lines rather than 8, which is what limits a stride-4 stem.  A
//    thread holds KRUN*4/BK pixels and reads its taps' table entries per lane.
//  kGatherStridedMask: the strided layout with padding, for filters of at
//    most 63 taps: entries are offset << 6 | tap, and each pixel holds a
//    64-bit mask of its taps outside the image (bit 63: past the reduction).
constexpr int kGatherScalar = 0, kGatherMask = 1, kGatherNoPad = 2, kGatherStrided = 3, kGatherStridedMask = 4;

// Bit r*S + s set for each tap (r, s) of a filter at input corner (h0, w0)
// that falls outside the H x W image: one row pattern (the columns outside)
// per filter row, or the whole row when the row itself is outside.  Needs
// R*S below the width of T.
template <typename T>
__device__ inline T outside_taps(int h0, int w0, int H, int W, int R, int S) {
    const int lo = max(0, -w0), hi = min(S, W - w0);  // columns s in [lo, hi) are inside
    const T row = (T(1) << S) - 1;
    const T inside = hi > lo ? (((T(1) << hi) - 1) & ~((T(1) << lo) - 1)) : T(0);
    const T cols_out = row & ~inside;
    T bad = 0;
    for (int r = 0; r < R; ++r)
        bad |= ((unsigned)(h0 + r) >= (unsigned)H ? row : cols_out) << (r * S);
    return bad;
}

// KS > 1: the workgroup holds KS groups of WMW x WNW waves that reduce
// interleaved slabs (group g takes slabs g, g + KS, ...) into the same
// output tile; their partial tiles are summed through LDS before the
// epilogue.  This gives small-pixel-count layers more waves without
// shrinking each wave's tile.
// The strided gathers ask the compiler for four waves per SIMD (at most 128
// registers a wave) where the tile allows it: up to three 32x32 accumulator
// blocks with 16-tap slabs, or one with 32-tap slabs; larger strided tiles
// cannot fit four and keep the compiler's default.
template <int WMW, int WNW, int FM, int FN, int BK, bool VEC_W, int GATHER, int KS, int ST>
__global__ void __launch_bounds__(64 * WMW * WNW * KS)
__attribute__((amdgpu_waves_per_eu(GATHER == kGatherStrided && FM * FN * BK <= 48 ? 4 : 1)))
conv2d_igemm_f32(ConvParams p) {
    static_assert(ST % 2 == 0, "the two LDS buffers alternate within a round of ST slabs");
    constexpr int TM = WMW * FM * 32;  // output channels per workgroup
    constexpr int TN = WNW * FN * 32;  // output pixels per workgroup
    constexpr int NT = 64 * WMW * WNW;  // threads per slab group
    constexpr int NTB = NT * KS;        // threads per workgroup
    constexpr int LDK = BK + 4;        // padded LDS row (conflict-free 128-bit reads)
    constexpr int KGROUPS = NT / TN;   // threads sharing one pixel column of the gather
    constexpr int KRUN = BK / KGROUPS; // consecutive taps gathered per thread
    static_assert(NT % TN == 0 && TN % 64 == 0, "gather layout needs TN | NT and whole waves per pixel column");
    static_assert(BK % KGROUPS == 0 && KRUN % 4 == 0, "gather run must be whole float4s");
    static_assert(BK % 8 == 0, "slab must split into two halves of float4s");
    constexpr int WTOT = VEC_W ? TM * BK / 4 : TM * BK;  // weight-tile loads per slab
    constexpr int WV = (WTOT + NT - 1) / NT;                // ... per thread
    constexpr int AROWS = WV * NT / (VEC_W ? BK / 4 : BK);  // TM rows + spare rows

    // LDS: [buffer][group] weight tiles [k][kk], then [buffer][group] im2col
    // tiles [m][kk]; reused at the end for the groups' partial tiles
    constexpr int A_ELEMS = AROWS * LDK, B_ELEMS = TN * LDK;
    __shared__ __attribute__((aligned(16))) float smem[2 * KS * (A_ELEMS + B_ELEMS)];
    static_assert((KS - 1) * TM * TN <= 2 * KS * (A_ELEMS + B_ELEMS), "reduction space");

    const int tid = threadIdx.x % NT;                                   // thread within its group
    const int sgrp = KS > 1 ? __builtin_amdgcn_readfirstlane(threadIdx.x / NT) : 0;  // slab group
    auto sA = [&](int buf) { return smem + (buf * KS + sgrp) * A_ELEMS; };
    auto sB = [&](int buf) { return smem + 2 * KS * A_ELEMS + (buf * KS + sgrp) * B_ELEMS; };
    const int g = blockIdx.z % p.G;
    const int kbeg = (blockIdx.z / p.G) * p.kchunk;  // first tap of this chunk
    const int klen = min(p.kchunk, p.Kr - kbeg);      // taps in this chunk
    // Workgroup -> tile.  A launch's workgroups go to the 8 XCDs in turn by
    // linear id, and each XCD has its own L2: the tiles that read the same
    // input (every channel tile of a pixel tile, and neighbouring pixel
    // tiles, whose windows overlap) are given to workgroups of one XCD, in
    // channel-tile-fastest order.  Ids past the last multiple of 8 keep their
    // position.
    int m0, k0;
    {
        const int gy = gridDim.y;
        const int tiles = gridDim.x * gy;
        const int wg = blockIdx.x + gridDim.x * blockIdx.y;
        const int full = tiles & ~7;
        const int seq = wg < full ? (wg & 7) * (full >> 3) + (wg >> 3) : wg;
        m0 = (seq / gy) * TN;
        k0 = (seq % gy) * TM;
    }

    // ---- gather setup: this thread's pixel and tap run (fixed for all slabs)
    const int mloc = tid % TN;
    const int kgrp = __builtin_amdgcn_readfirstlane(tid / TN);  // uniform: TN is a multiple of 64
    const int m = m0 + mloc;
    int hb, wb, lane_off;
    if (m < p.M) {
        const int n = (int)fdiv(m, p.f_pq);
        const int pq = m - n * p.PQ;
        const int pp = (int)fdiv(pq, p.f_q);
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

    const int nslab = (klen + BK - 1) / BK;
    const int niter = (nslab + KS - 1) / KS;  // slabs per group
    extern __shared__ __attribute__((aligned(16))) int stab[];  // (niter + ST) * KS * BK entries
    unsigned inv = 0xffffffffu;
    if constexpr (GATHER != kGatherScalar) {
        for (int kk = threadIdx.x; kk < (niter + ST) * KS * BK; kk += NTB) {
            int e = GATHER == kGatherMask ? 31 : GATHER == kGatherStridedMask ? 63 : (int)0x80000000u;
            if (kk < klen) {
                const int c = (int)fdiv(kbeg + kk, p.f_rs);
                const int rs = kbeg + kk - c * p.RS;
                const int r = (int)fdiv(rs, p.f_s);
                const int s = rs - r * p.S;
                const int toff = ((c * p.H + r) * p.W + s) * 4;
                e = GATHER == kGatherMask ? ((toff << 5) | rs) : GATHER == kGatherStridedMask ? ((toff << 6) | rs) : toff;
            }
            stab[kk] = e;
        }
        if (GATHER == kGatherNoPad && m >= p.M) lane_off = (int)0x80000000u;
    }
    if constexpr (GATHER == kGatherMask) {
        if (m < p.M) inv = 0x80000000u | outside_taps<unsigned>(hb, wb, p.H, p.W, p.R, p.S);
    }
    // strided gather: element u of a thread is pixel group u / TG (16 pixels
    // apart) and tap group u % TG (4 taps apart) of its wave's pixels
    constexpr int TG = BK / 4;          // tap groups per slab
    constexpr int PPT = KRUN / TG;      // pixels per thread
    constexpr int PW = 16 * PPT;        // pixels per wave
    constexpr bool STRIDED = GATHER == kGatherStrided || GATHER == kGatherStridedMask;
    static_assert(!STRIDED || (KRUN % TG == 0 && (NT / 64) * PW == TN),
                  "strided gather: whole pixel groups per wave");
    const int ln = tid & 63;
    const int wpix = (tid >> 6) * PW + (ln >> 2);  // this thread's first pixel, within the tile
    int soff[STRIDED ? PPT : 1];
    unsigned long long inv64[GATHER == kGatherStridedMask ? PPT : 1];
    if constexpr (STRIDED) {
#pragma unroll
        for (int pi = 0; pi < PPT; ++pi) {
            const int mm = m0 + wpix + pi * 16;
            inv64[GATHER == kGatherStridedMask ? pi : 0] = ~0ull;
            if (mm < p.M) {
                const int n = (int)fdiv(mm, p.f_pq);
                const int pq = mm - n * p.PQ;
                const int pp = (int)fdiv(pq, p.f_q);
                const int qq = pq - pp * p.Q;
                const int h0 = pp * p.sh - p.ph, w0 = qq * p.sw - p.pw;
                soff[pi] = ((n * p.C + g * p.Cg) * p.HW + h0 * p.W + w0) * 4;
                if constexpr (GATHER == kGatherStridedMask)
                    inv64[pi] = (1ull << 63) | outside_taps<unsigned long long>(h0, w0, p.H, p.W, p.R, p.S);
            } else {
                soff[pi] = GATHER == kGatherStridedMask ? 0 : (int)0x80000000u;
            }
        }
    }
    if constexpr (GATHER != kGatherScalar) __syncthreads();

    float xr[ST][KRUN];  // register stages
    auto load_x = [&](int kslab, int sg) {
        if constexpr (STRIDED) {
#pragma unroll
            for (int q = 0; q < TG; ++q) {
                const int e = stab[kslab + 4 * q + (ln & 3)];
#pragma unroll
                for (int pi = 0; pi < PPT; ++pi) {
                    int voff;
                    if constexpr (GATHER == kGatherStridedMask) {
                        const unsigned bad = (unsigned)(inv64[pi] >> (e & 63)) & 1u;
                        voff = (soff[pi] + (e >> 6)) | (int)(bad << 31);
                    } else {
                        voff = (int)((unsigned)soff[pi] + (unsigned)e);
                    }
                    xr[sg][pi * TG + q] =
                        __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, voff, 0, 0));
                }
            }
            return;
        }
        const int kk0 = kslab + kgrp * KRUN;  // uniform
        if constexpr (GATHER != kGatherScalar) {
#pragma unroll
            for (int j = 0; j < KRUN; j += 4) {
                const int4 e4 = *reinterpret_cast<const int4*>(&stab[kk0 + j]);
                const int es[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    int voff;
                    if constexpr (GATHER == kGatherMask) {
                        const unsigned bad = (inv >> (es[u] & 31)) & 1u;
                        voff = (lane_off + (int)((unsigned)es[u] >> 5)) | (int)(bad << 31);
                    } else {
                        voff = (int)((unsigned)lane_off + (unsigned)es[u]);
                    }
                    xr[sg][j + u] =
                        __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, voff, 0, 0));
                }
            }
            return;
        }
        const int ka0 = kbeg + kk0;  // absolute tap index
        int c = (int)fdiv(ka0, p.f_rs);
        const int rs = ka0 - c * p.RS;
        int r = (int)fdiv(rs, p.f_s);
        int s = rs - r * p.S;
        int toff = ((c * p.H + r) * p.W + s) * 4;  // byte offset of tap (c, r, s)
#pragma unroll
        for (int j = 0; j < KRUN; ++j) {
            const bool ok = (kk0 + j < klen) && ((unsigned)(hb + r) < (unsigned)p.H) &&
                            ((unsigned)(wb + s) < (unsigned)p.W);
            const int voff = ok ? lane_off + toff : kOutOfRange;
            xr[sg][j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xres, voff, 0, 0));
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
    auto store_x = [&](int buf, int sg) {
        if (p.relu_x) {  // uniform
#pragma unroll
            for (int j = 0; j < KRUN; ++j) xr[sg][j] = xr[sg][j] > 0.0f ? xr[sg][j] : 0.0f;
        }
        if constexpr (STRIDED) {
            float* dst = sB(buf) + wpix * LDK + (ln & 3);
#pragma unroll
            for (int u = 0; u < KRUN; ++u) dst[(u / TG) * 16 * LDK + 4 * (u % TG)] = xr[sg][u];
            return;
        }
        float* dst = sB(buf) + mloc * LDK + kgrp * KRUN;
#pragma unroll
        for (int j = 0; j < KRUN; j += 4)
            *reinterpret_cast<float4*>(dst + j) =
                make_float4(xr[sg][j], xr[sg][j + 1], xr[sg][j + 2], xr[sg][j + 3]);
    };

    // ---- weight tile loads: rows k0.. of the group's [Kg][Kr] block, through a
    // buffer resource as well (rows past the group or taps past the reduction
    // read as zero).  Items past the tile land in spare LDS rows never read.
    const __amdgpu_buffer_rsrc_t wres =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p.w), (short)0, p.wbytes, 0x00020000);
    constexpr int VW = VEC_W ? 4 : 1;
    int w_off[WV], w_col[WV], w_lds[WV];
    bool w_rowok[WV];
#pragma unroll
    for (int i = 0; i < WV; ++i) {
        const int idx = tid + i * NT;
        const int row = idx / (BK / VW);
        w_col[i] = (idx % (BK / VW)) * VW;
        w_rowok[i] = row < TM && k0 + row < p.Kg;
        w_off[i] = w_rowok[i] ? ((g * p.Kg + k0 + row) * p.Kr + kbeg + w_col[i]) * 4 : 0;
        w_lds[i] = row * LDK + w_col[i];
    }
    float wr[ST][WV * VW];
    auto load_w = [&](int kslab, int sg) {
#pragma unroll
        for (int i = 0; i < WV; ++i) {
            if constexpr (VEC_W) {
                const bool ok = w_rowok[i] && (kslab + w_col[i] < klen);
                const int voff = ok ? w_off[i] + kslab * 4 : kOutOfRange;
                // Cast the whole vector: a bit-cast of one element of an
                // ext_vector lvalue reads element 0 with this compiler.
                typedef float f32x4 __attribute__((ext_vector_type(4)));
                const f32x4 v =
                    __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(wres, voff, 0, 0));
                wr[sg][4 * i] = v[0];
                wr[sg][4 * i + 1] = v[1];
                wr[sg][4 * i + 2] = v[2];
                wr[sg][4 * i + 3] = v[3];
            } else {
                const bool ok = w_rowok[i] && (kslab + w_col[i] < klen);
                const int voff = ok ? w_off[i] + kslab * 4 : kOutOfRange;
                wr[sg][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(wres, voff, 0, 0));
            }
        }
    };
    auto store_w = [&](int buf, int sg) {
#pragma unroll
        for (int i = 0; i < WV; ++i) {
            if constexpr (VEC_W)
                *reinterpret_cast<float4*>(sA(buf) + w_lds[i]) =
                    make_float4(wr[sg][4 * i], wr[sg][4 * i + 1], wr[sg][4 * i + 2], wr[sg][4 * i + 3]);
            else
                sA(buf)[w_lds[i]] = wr[sg][i];
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
            const float* src = sA(buf) + (wm * FM * 32 + i * 32 + l32) * LDK + half * (BK / 2);
#pragma unroll
            for (int t = 0; t < BK / 2; t += 4) {
                const float4 v = *reinterpret_cast<const float4*>(src + t);
                a[i][t] = v.x; a[i][t + 1] = v.y; a[i][t + 2] = v.z; a[i][t + 3] = v.w;
            }
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const float* src = sB(buf) + (wn * FN * 32 + j * 32 + l32) * LDK + half * (BK / 2);
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

    // ---- main loop: slab s computes from LDS while slabs s+1 .. s+ST load.
    // ST slabs of loads in flight (ST register stages).  Slab s is stored to
    // LDS buffer s % 2 from register stage s % ST, then slab s + ST is
    // requested into that stage and slab s is multiplied.  One barrier per
    // slab, which also guarantees that nobody still reads the buffer for slab
    // s - 2.  The last niter % ST slabs run after the loop, so that the loop
    // body is straight-line code and each store waits only for its own slab's
    // loads.
    auto slab_k = [&](int it) { return (it * KS + sgrp) * BK; };  // first tap of group slab it
#pragma unroll
    for (int j = 0; j < ST; ++j) {
        load_x(slab_k(j), j);
        load_w(slab_k(j), j);
    }
    int it = 0;
    for (; it + ST - 1 < niter; it += ST) {
#pragma unroll
        for (int j = 0; j < ST; ++j) {
            store_x(j & 1, j);
            store_w(j & 1, j);
            __syncthreads();
            load_x(slab_k(it + j + ST), j);
            load_w(slab_k(it + j + ST), j);
            compute(j & 1);
            if constexpr (!STRIDED) {
                // Instruction order within the slab: the fragment reads, then
                // the matrix-core instructions with one of the next slabs'
                // global loads after each, rather than all loads ahead of the
                // reads.  Measured on AlexNet at batch 64: conv2/conv3 3-5%
                // faster than the compiler's order; one load per two
                // instructions, or two per instruction, was slower.  The
                // strided gathers keep the compiler's order: pinned, the
                // 512-thread tiles returned zeros for the last tap of every
                // other slab in the last lanes of a wave whenever two
                // workgroups shared a compute unit (the last gather load of
                // the slab read a reused address register); the compiler's
                // order gave exact results, at 3% on the stride-4 stem
                // (AlexNet conv1 at batch 64: 132 -> 136 us).
                constexpr int NR = (FM + FN) * (BK / 8);  // fragment reads
                constexpr int NM = FM * FN * (BK / 2);    // matrix-core instructions
                constexpr int NL = KRUN + WV;             // global loads
                __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);  // LDS reads
#pragma unroll
                for (int q = 0; q < NM; ++q) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                    if (q < NL) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
                }
            }
        }
    }
#pragma unroll
    for (int j = 0; j < ST - 1; ++j) {
        if (it + j < niter) {
            store_x(j & 1, j);
            store_w(j & 1, j);
            __syncthreads();
            compute(j & 1);
        }
    }
    if constexpr (KS > 1) __syncthreads();  // the group reduction reuses the tile buffers

    // ---- sum the slab groups' partial tiles (lanes on consecutive words)
    if constexpr (KS > 1) {
        constexpr int E = FM * FN * 16;
        if (sgrp > 0) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        smem[((sgrp - 1) * E + (i * FN + j) * 16 + v) * NT + tid] = acc[i][j][v];
        }
        __syncthreads();
        if (sgrp > 0) return;
#pragma unroll
        for (int q = 1; q < KS; ++q)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        acc[i][j][v] += smem[((q - 1) * E + (i * FN + j) * 16 + v) * NT + tid];
    }

    // ---- epilogue: bias, ReLU, NCHW store (lanes = consecutive pixels).  The
    // FN pixel blocks of one output channel are stored one after the other,
    // so that a channel's run of FN * 32 pixels reaches L2 in consecutive
    // instructions (with the blocks stored far apart, 128 x 128 tiles on
    // planes that are not a whole number of cache lines wrote 1.36x their
    // output to HBM: partial lines written back separately).
    float* yb[FN];
    bool mok[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int mc = m0 + wn * FN * 32 + j * 32 + l32;
        mok[j] = mc < p.M;
        const int n = mok[j] ? (int)fdiv(mc, p.f_pq) : 0;
        const int pq = mok[j] ? mc - n * p.PQ : 0;
        yb[j] = p.y + n * p.K * p.PQ + pq;
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int kr = k0 + wm * FM * 32 + i * 32 + 8 * (v / 4) + 4 * half + (v % 4);
            if (kr >= p.Kg) continue;
            const int ko = g * p.Kg + kr;
            const float bv = (p.splits == 1 && p.bias) ? p.bias[ko] : 0.0f;
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                if (!mok[j]) continue;
                float val = acc[i][j][v];
                if (p.splits > 1) {
                    atomicAdd(yb[j] + ko * p.PQ, val);
                } else {
                    if (p.bias) val += bv;
                    if (p.relu) val = val > 0.0f ? val : 0.0f;
                    yb[j][ko * p.PQ] = val;
                }
            }
        }
    }
}

// ---------------------------------------------------------------- configurations
typedef int (*LaunchFn)(const ConvParams&, bool vec_w, hipStream_t st);

template <int WMW, int WNW, int FM, int FN, int BK, int KS, int ST, bool VEC_W, int GATHER>
inline void launch_kernel(const ConvParams& prm, dim3 grid, dim3 block, size_t shm, hipStream_t st) {
    enqueue((conv2d_igemm_f32<WMW, WNW, FM, FN, BK, VEC_W, GATHER, KS, ST>), grid, block, shm, st, prm);
}

// Picks the gather mode for the shape and launches one configuration.
template <int WMW, int WNW, int FM, int FN, int BK, int KS, int ST>
int launch_cfg(const ConvParams& prm, bool vec_w, hipStream_t st) {
    constexpr int TM = WMW * FM * 32;
    constexpr int TN = WNW * FN * 32;
    dim3 grid(ceil_div(prm.M, TN), ceil_div(prm.Kg, TM), prm.G * prm.splits);
    dim3 block(64 * WMW * WNW * KS);
    // tap tables are at most 32 KiB of LDS
    const int tab_entries = (ceil_div(ceil_div(prm.kchunk, BK), KS) + ST) * KS * BK;
    const bool tab_fits = tab_entries * 4 <= 32768;
    int mode = kGatherScalar;
    if (tab_fits && prm.ph == 0 && prm.pw == 0)
        mode = prm.sw > 1 ? kGatherStrided : kGatherNoPad;
    else if (tab_fits && prm.sw > 1 && prm.RS <= 63 && (int64_t)prm.Cg * prm.HW * 4 < ((int64_t)1 << 25))
        mode = kGatherStridedMask;
    else if (tab_fits && prm.RS <= 31 && (int64_t)prm.Cg * prm.HW * 4 < ((int64_t)1 << 27))
        mode = kGatherMask;
    const size_t shm = mode == kGatherScalar ? 0 : (size_t)tab_entries * 4;
    if (vec_w) {
        if (mode == kGatherStridedMask) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, true, kGatherStridedMask>(prm, grid, block, shm, st);
        else if (mode == kGatherStrided) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, true, kGatherStrided>(prm, grid, block, shm, st);
        else if (mode == kGatherNoPad) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, true, kGatherNoPad>(prm, grid, block, shm, st);
        else if (mode == kGatherMask) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, true, kGatherMask>(prm, grid, block, shm, st);
        else launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, true, kGatherScalar>(prm, grid, block, shm, st);
    } else {
        if (mode == kGatherStridedMask) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, false, kGatherStridedMask>(prm, grid, block, shm, st);
        else if (mode == kGatherStrided) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, false, kGatherStrided>(prm, grid, block, shm, st);
        else if (mode == kGatherNoPad) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, false, kGatherNoPad>(prm, grid, block, shm, st);
        else if (mode == kGatherMask) launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, false, kGatherMask>(prm, grid, block, shm, st);
        else launch_kernel<WMW, WNW, FM, FN, BK, KS, ST, false, kGatherScalar>(prm, grid, block, shm, st);
    }
    return check_launch("conv2d_igemm_f32");
}

// The configurations: index, waves along output channels, waves along
// pixels, 32x32 blocks per wave along channels and pixels, slab length,
// slab groups per workgroup, register stages of slabs in flight.
#define CNN_CONV_CONFIGS(X)      \
    X(0, 2, 2, 2, 2, 16, 1, 2)  /* 128 x 128 */  \
    X(1, 2, 2, 2, 2, 32, 1, 2)  /* 128 x 128 */  \
    X(2, 4, 1, 1, 2, 16, 1, 2)  /* 128 x 64 */   \
    X(3, 4, 1, 1, 2, 32, 1, 2)  /* 128 x 64 */   \
    X(4, 1, 4, 2, 1, 16, 1, 2)  /* 64 x 128 */   \
    X(5, 1, 4, 2, 1, 32, 1, 2)  /* 64 x 128 */   \
    X(6, 1, 4, 3, 1, 16, 1, 2)  /* 96 x 128 */   \
    X(7, 1, 4, 3, 1, 32, 1, 2)  /* 96 x 128 */   \
    X(8, 1, 4, 1, 1, 16, 1, 2)  /* 32 x 128 */   \
    X(9, 2, 2, 1, 1, 16, 1, 2)  /* 64 x 64 */    \
    X(10, 2, 2, 1, 1, 32, 1, 2) /* 64 x 64 */    \
    X(11, 2, 4, 2, 2, 16, 1, 2) /* 128 x 256, 8 waves */ \
    X(12, 1, 2, 3, 2, 16, 1, 2) /* 96 x 128, 2 waves */  \
    X(13, 2, 1, 2, 2, 16, 1, 2) /* 128 x 64, 2 waves */  \
    X(14, 2, 2, 1, 1, 16, 2, 2) /* 64 x 64, 2 slab groups of 4 waves */  \
    X(15, 2, 1, 2, 2, 16, 2, 2) /* 128 x 64, 2 slab groups of 2 waves */

#define CNN_CONV_DECLARE(I, WMW, WNW, FM, FN, BK, KS, ST) \
    int launch_c##I(const ConvParams& prm, bool vec_w, hipStream_t st);
CNN_CONV_CONFIGS(CNN_CONV_DECLARE)

// Defines launch_c<I> (one translation unit per group of configurations).
#define CNN_CONV_DEFINE(I, WMW, WNW, FM, FN, BK, KS, ST)                           \
    int launch_c##I(const ConvParams& prm, bool vec_w, hipStream_t st) {           \
        return launch_cfg<WMW, WNW, FM, FN, BK, KS, ST>(prm, vec_w, st);           \
    }

}  // namespace conv
}  // namespace cnn
