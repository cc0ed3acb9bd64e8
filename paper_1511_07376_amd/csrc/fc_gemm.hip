// Fully-connected layer on the fp32 matrix cores of gfx950.
//
//     Y[n][o] = b[o] + sum_i X[n][i] * W[o][i]
//
// Both operands are stored with the reduction index contiguous ([N][I] and
// [O][I]), so the workgroup stages a TM x BK slab of X and a TN x BK slab of
// W in LDS with 128-bit loads.  The image index is the MFMA row and the
// output feature the MFMA column: the 32 lanes of a row write 32 consecutive
// outputs.  A batch of 16 to 256 images gives few output tiles, far fewer
// than the chip's 256 compute units, so the reduction is split across
// workgroups (grid z); the partial sums are added with fp32 atomics into an
// output pre-filled with the bias, and a ReLU, when the layer has one, runs
// after the last partial sum has landed.
#include "common.h"

#include <algorithm>

namespace cnn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

struct FcParams {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int N, I, O;
    int kchunk;  // reduction length per split (multiple of BK)
    int relu;
};

// Loads rows [r0, r0 + tile rows) x columns [kslab, kslab + BK) of a row-major
// matrix with leading dimension ld into registers, zero outside rows_total
// and kend.  Thread tid takes items tid, tid + NT, ... of the tile.
template <int NVEC, int TOT, int NT, int BK, bool VEC>
__device__ inline void load_tile(const float* base, int ld, int rows_total, int r0, int kslab,
                                 int kend, int tid, float* reg) {
    constexpr int VW = VEC ? 4 : 1;
#pragma unroll
    for (int i = 0; i < NVEC; ++i) {
        const int idx = tid + i * NT;
        if (TOT % NT != 0 && idx >= TOT) break;
        const int row = idx / (BK / VW);
        const int col = (idx % (BK / VW)) * VW;
        const int gr = r0 + row, kk = kslab + col;
        if constexpr (VEC) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (gr < rows_total && kk < kend)
                v = *reinterpret_cast<const float4*>(base + (size_t)gr * ld + kk);
            reg[4 * i] = v.x; reg[4 * i + 1] = v.y; reg[4 * i + 2] = v.z; reg[4 * i + 3] = v.w;
        } else {
            reg[i] = (gr < rows_total && kk < kend) ? base[(size_t)gr * ld + kk] : 0.0f;
        }
    }
}

template <int NVEC, int TOT, int NT, int BK, int LDK, bool VEC>
__device__ inline void store_tile(float* dst, int tid, const float* reg) {
    constexpr int VW = VEC ? 4 : 1;
#pragma unroll
    for (int i = 0; i < NVEC; ++i) {
        const int idx = tid + i * NT;
        if (TOT % NT != 0 && idx >= TOT) break;
        const int row = idx / (BK / VW);
        const int col = (idx % (BK / VW)) * VW;
        if constexpr (VEC)
            *reinterpret_cast<float4*>(dst + row * LDK + col) =
                make_float4(reg[4 * i], reg[4 * i + 1], reg[4 * i + 2], reg[4 * i + 3]);
        else
            dst[row * LDK + col] = reg[i];
    }
}

template <int WMW, int WNW, int FM, int FN, int BK, bool VEC, bool SPLIT>
__global__ void __launch_bounds__(64 * WMW * WNW)
fc_gemm_f32(FcParams p) {
    constexpr int TM = WMW * FM * 32;  // images per workgroup
    constexpr int TN = WNW * FN * 32;  // output features per workgroup
    constexpr int NT = 64 * WMW * WNW;
    constexpr int LDK = BK + 4;
    constexpr int VW = VEC ? 4 : 1;                // floats per load
    constexpr int ATOT = TM * BK / VW, BTOT = TN * BK / VW;
    constexpr int AV = (ATOT + NT - 1) / NT, BV = (BTOT + NT - 1) / NT;
    static_assert(BK % 8 == 0, "slab must split into two halves of float4s");

    __shared__ __attribute__((aligned(16))) float sA[2][TM * LDK];  // X [n][i]
    __shared__ __attribute__((aligned(16))) float sB[2][TN * LDK];  // W [o][i]

    const int tid = threadIdx.x;
    const int n0 = blockIdx.y * TM;
    const int o0 = blockIdx.x * TN;
    const int kbeg = blockIdx.z * p.kchunk;
    const int kend = min(p.I, kbeg + p.kchunk);

    float ra[AV * VW], rb[BV * VW];

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

    const int nslab = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
    if (nslab > 0) {
        load_tile<AV, ATOT, NT, BK, VEC>(p.x, p.I, p.N, n0, kbeg, kend, tid, ra);
        load_tile<BV, BTOT, NT, BK, VEC>(p.w, p.I, p.O, o0, kbeg, kend, tid, rb);
        store_tile<AV, ATOT, NT, BK, LDK, VEC>(sA[0], tid, ra);
        store_tile<BV, BTOT, NT, BK, LDK, VEC>(sB[0], tid, rb);
        __syncthreads();
    }
    for (int sl = 0; sl < nslab; ++sl) {
        const int cur = sl & 1;
        const bool more = sl + 1 < nslab;
        if (more) {
            load_tile<AV, ATOT, NT, BK, VEC>(p.x, p.I, p.N, n0, kbeg + (sl + 1) * BK, kend, tid, ra);
            load_tile<BV, BTOT, NT, BK, VEC>(p.w, p.I, p.O, o0, kbeg + (sl + 1) * BK, kend, tid, rb);
        }
        compute(cur);
        if (more) {
            store_tile<AV, ATOT, NT, BK, LDK, VEC>(sA[cur ^ 1], tid, ra);
            store_tile<BV, BTOT, NT, BK, LDK, VEC>(sB[cur ^ 1], tid, rb);
        }
        __syncthreads();
    }

#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int o = o0 + wn * FN * 32 + j * 32 + l32;
        if (o >= p.O) continue;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int n = n0 + wm * FM * 32 + i * 32 + 8 * (v / 4) + 4 * half + (v % 4);
                if (n < p.N) {
                    float* dst = p.y + (size_t)n * p.O + o;
                    if constexpr (SPLIT) {
                        atomicAdd(dst, acc[i][j][v]);
                    } else {
                        float val = acc[i][j][v];
                        if (p.bias) val += p.bias[o];
                        if (p.relu) val = val > 0.0f ? val : 0.0f;
                        *dst = val;
                    }
                }
            }
        }
    }
}

// y[n][o] = bias[o] (or 0): the starting value of the split-reduction sums.
__global__ void fc_fill_bias(float* y, const float* bias, int N, int O) {
    const int total = N * O;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x)
        y[i] = bias ? bias[i % O] : 0.0f;
}

template <int WMW, int WNW, int FM, int FN, int BK>
int launch_fc_cfg(const FcParams& prm0, bool vec, hipStream_t st) {
    constexpr int TM = WMW * FM * 32;
    constexpr int TN = WNW * FN * 32;
    FcParams prm = prm0;
    const int tiles = ceil_div(prm.N, TM) * ceil_div(prm.O, TN);
    // Enough workgroups to cover the 256 compute units about twice, but keep
    // at least four slabs of reduction per workgroup.
    int splits = ceil_div(512, tiles);
    const int max_splits = std::max(1, prm.I / (4 * BK));
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    prm.kchunk = ceil_div(ceil_div(prm.I, splits), BK) * BK;
    splits = ceil_div(prm.I, prm.kchunk);
    dim3 grid(ceil_div(prm.O, TN), ceil_div(prm.N, TM), splits);
    dim3 block(64 * WMW * WNW);
    if (splits > 1) {
        const int total = prm.N * prm.O;
        hipLaunchKernelGGL(fc_fill_bias, dim3(std::min(ceil_div(total, 256), 2048)), dim3(256), 0, st,
                           prm.y, prm.bias, prm.N, prm.O);
        if (vec)
            hipLaunchKernelGGL((fc_gemm_f32<WMW, WNW, FM, FN, BK, true, true>), grid, block, 0, st, prm);
        else
            hipLaunchKernelGGL((fc_gemm_f32<WMW, WNW, FM, FN, BK, false, true>), grid, block, 0, st, prm);
        int rc = check_launch("fc_gemm_f32");
        if (rc != CNN_OK) return rc;
        if (prm.relu) return launch_relu(prm.y, prm.y, (int64_t)prm.N * prm.O, st);
        return CNN_OK;
    }
    if (vec)
        hipLaunchKernelGGL((fc_gemm_f32<WMW, WNW, FM, FN, BK, true, false>), grid, block, 0, st, prm);
    else
        hipLaunchKernelGGL((fc_gemm_f32<WMW, WNW, FM, FN, BK, false, false>), grid, block, 0, st, prm);
    return check_launch("fc_gemm_f32");
}

}  // namespace

int launch_fc(const float* x, int N, int I, const float* w, const float* bias, int O, int relu,
              float* y, hipStream_t st) {
    if (N == 0) return CNN_OK;
    FcParams prm;
    prm.x = x;
    prm.w = w;
    prm.bias = bias;
    prm.y = y;
    prm.N = N;
    prm.I = I;
    prm.O = O;
    prm.kchunk = I;
    prm.relu = relu;
    const bool vec = (I % 4 == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0) &&
                     ((reinterpret_cast<uintptr_t>(w) & 15) == 0);
    if (N <= 32) return launch_fc_cfg<1, 4, 1, 1, 32>(prm, vec, st);   // 32 x 128
    if (N <= 64) return launch_fc_cfg<1, 4, 2, 1, 32>(prm, vec, st);   // 64 x 128
    return launch_fc_cfg<2, 2, 2, 2, 16>(prm, vec, st);                // 128 x 128
}

}  // namespace cnn
