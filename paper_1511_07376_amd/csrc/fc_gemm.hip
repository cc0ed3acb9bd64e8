// Fully-connected layer on the fp32 matrix cores of gfx950.
//
//     Y[n][o] = b[o] + sum_i X[n][i] * W[o][i]
//
// Both operands are stored with the reduction index contiguous ([N][I] and
// [O][I]), so the workgroup stages a TM x BK slab of X and a TN x BK slab of
// W in LDS with 128-bit loads.  The image index is the MFMA row and the
// output feature the MFMA column: the 32 lanes of a row write 32 consecutive
// outputs.
//
// W is read exactly once and comes from HBM, far away in latency compared
// with the matrix-core time of one slab, so each thread keeps D slabs of loads
// in flight in a register ring (slab s + D + 1 is requested as slab s + 1 is
// stored to LDS).  The LDS round trip of a slab (store, barrier, fragment
// reads) overlaps the matrix-core work of the slab before it: a wave holds
// two sets of fragment registers, and the barrier that publishes slab s + 1
// sits inside slab s's matrix-core instructions.  The loads go through buffer
// resources: an index past the matrix gets an out-of-range offset that reads
// 0, so the loads carry no branches and the compiler can wait for exactly the
// slab it needs rather than for all of them.
//
// A batch of 1 to 256 images gives few output tiles, far fewer than the
// chip's 256 compute units, so the reduction is split across workgroups
// (grid z); the partial sums are added with fp32 atomics into an output
// pre-filled with the bias, and a ReLU, when the layer has one, runs after the
// last partial sum has landed.
#include "common.h"
#include "fill_jobs.h"

#include <algorithm>
#include <type_traits>

namespace cnn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kOutOfRange = (int)0x80000000u;  // buffer offset that reads as 0

struct FcParams {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int N, I, O;
    int kchunk;  // reduction length per split (a multiple of D * BK)
    int relu;
};

// Loads rows [0, rows) x columns [kslab, kslab + BK) of the row-major matrix
// behind `rs` (leading dimension ld; columns past kend and rows past `rows`
// read as 0) into registers.  Thread tid takes items tid, tid + NT, ... of
// VW floats (4: 128-bit loads, which need ld and the bases 16-byte aligned).
template <int NVEC, int TOT, int NT, int BK, int VW>
__device__ inline void load_tile(__amdgpu_buffer_rsrc_t rs, int ld, int rows, int kslab, int kend,
                                 int tid, float* reg) {
#pragma unroll
    for (int i = 0; i < NVEC; ++i) {
        const int idx = tid + i * NT;
        const int row = idx / (BK / VW);
        const int kk = kslab + (idx % (BK / VW)) * VW;
        const bool ok = (TOT % NT == 0 || idx < TOT) && row < rows && kk < kend;
        const int voff = ok ? (row * ld + kk) * 4 : kOutOfRange;
        if constexpr (VW == 4) {
            // Cast the whole vector: a bit-cast of one element of an
            // ext_vector lvalue reads element 0 with this compiler.
            const f32x4 v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, 0, 0));
            reg[4 * i] = v[0];
            reg[4 * i + 1] = v[1];
            reg[4 * i + 2] = v[2];
            reg[4 * i + 3] = v[3];
        } else {
            reg[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, 0, 0));
        }
    }
}

// RELU: store max(v, 0) (the input of a layer whose producer's ReLU was
// deferred to its consumer).
template <int NVEC, int TOT, int NT, int BK, int LDK, int VW, bool RELU = false>
__device__ inline void store_tile(float* dst, int tid, const float* reg) {
    auto r = [](float v) { return RELU ? (v > 0.0f ? v : 0.0f) : v; };
#pragma unroll
    for (int i = 0; i < NVEC; ++i) {
        const int idx = tid + i * NT;
        if (TOT % NT != 0 && idx >= TOT) break;
        const int row = idx / (BK / VW);
        const int col = (idx % (BK / VW)) * VW;
        if constexpr (VW == 4)
            *reinterpret_cast<float4*>(dst + row * LDK + col) =
                make_float4(r(reg[4 * i]), r(reg[4 * i + 1]), r(reg[4 * i + 2]), r(reg[4 * i + 3]));
        else
            dst[row * LDK + col] = r(reg[i]);
    }
}

// RELU_X: the layer's input is taken through a ReLU.
template <int WMW, int WNW, int FM, int FN, int BK, int D, bool VEC, bool SPLIT, bool RELU_X>
__global__ void __launch_bounds__(64 * WMW * WNW)
fc_gemm_f32(FcParams p) {
    constexpr int TM = WMW * FM * 32;  // images per workgroup
    constexpr int TN = WNW * FN * 32;  // output features per workgroup
    constexpr int NT = 64 * WMW * WNW;
    constexpr int LDK = BK + 4;        // padded LDS row (conflict-free 128-bit reads)
    constexpr int VW = VEC ? 4 : 1;    // floats per load
    constexpr int ATOT = TM * BK / VW, BTOT = TN * BK / VW;
    constexpr int AV = (ATOT + NT - 1) / NT, BV = (BTOT + NT - 1) / NT;
    static_assert(BK % 8 == 0, "slab must split into two halves of float4s");
    static_assert(D % 2 == 0, "the two LDS buffers alternate within a round of D slabs");

    __shared__ __attribute__((aligned(16))) float sA[2][TM * LDK];  // X [n][i]
    __shared__ __attribute__((aligned(16))) float sB[2][TN * LDK];  // W [o][i]

    const int tid = threadIdx.x;
    const int n0 = blockIdx.y * TM;
    const int o0 = blockIdx.x * TN;
    const int kbeg = blockIdx.z * p.kchunk;
    const int klen = min(p.I - kbeg, p.kchunk);  // this split's reduction length
    const int xrows = min(TM, p.N - n0);
    const int wrows = min(TN, p.O - o0);
    // resources based at this workgroup's first row and first tap
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(p.x + (size_t)n0 * p.I + kbeg), (short)0, 0x7fffffff, 0x00020000);
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(p.w + (size_t)o0 * p.I + kbeg), (short)0, 0x7fffffff, 0x00020000);

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

    // fragment set `set` <- the wave's rows of LDS buffer `buf`
    float fa[2][FM][BK / 2], fb[2][FN][BK / 2];
    auto read_frags = [&](int buf, int set) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const float* src = &sA[buf][(wm * FM * 32 + i * 32 + l32) * LDK + half * (BK / 2)];
#pragma unroll
            for (int t = 0; t < BK / 2; t += 4) {
                const float4 v = *reinterpret_cast<const float4*>(src + t);
                fa[set][i][t] = v.x; fa[set][i][t + 1] = v.y; fa[set][i][t + 2] = v.z; fa[set][i][t + 3] = v.w;
            }
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const float* src = &sB[buf][(wn * FN * 32 + j * 32 + l32) * LDK + half * (BK / 2)];
#pragma unroll
            for (int t = 0; t < BK / 2; t += 4) {
                const float4 v = *reinterpret_cast<const float4*>(src + t);
                fb[set][j][t] = v.x; fb[set][j][t + 1] = v.y; fb[set][j][t + 2] = v.z; fb[set][j][t + 3] = v.w;
            }
        }
    };
    // matrix-core instructions of k-steps [t0, t1) of the slab in fragment set `set`
    auto mfma = [&](int set, int t0, int t1) {
#pragma unroll
        for (int t = t0; t < t1; ++t)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[set][i][t], fb[set][j][t], acc[i][j], 0, 0, 0);
    };

    // Step s (slab s's fragments are in set s % 2, slab s + 1 in ring slot
    // (s + 1) % D): store slab s + 1 to LDS buffer (s + 1) % 2; issue the
    // first 3/4 of slab s's matrix-core instructions; barrier; read slab
    // s + 1's fragments into set (s + 1) % 2 and request slab s + 1 + D into
    // the freed ring slot; issue the rest of slab s's instructions.  Buffer
    // (s + 1) % 2 last held slab s - 1, whose fragments every wave consumed
    // before the barrier of step s - 1.  kchunk is a multiple of D * BK; only
    // the last split can end inside a round, where the slabs past its end
    // read as zeros (the steps past the last slab store and read zeros too).
    // Measured on AlexNet's FC shapes at batches 16, 64 and 256 (one
    // workgroup timed per wave): 3-13% faster than storing, synchronising and
    // reading each slab just before its own instructions; 1/2 or 3/4 of the
    // instructions before the barrier, and 32-tap slabs, within 2% of it.
    constexpr int H = 3 * BK / 8;  // k-steps before the barrier
    float ra[D][AV * VW], rb[D][BV * VW];
#pragma unroll
    for (int j = 0; j < D; ++j) {
        load_tile<AV, ATOT, NT, BK, VW>(xres, p.I, xrows, j * BK, klen, tid, ra[j]);
        load_tile<BV, BTOT, NT, BK, VW>(wres, p.I, wrows, j * BK, klen, tid, rb[j]);
    }
    store_tile<AV, ATOT, NT, BK, LDK, VW, RELU_X>(sA[0], tid, ra[0]);
    store_tile<BV, BTOT, NT, BK, LDK, VW>(sB[0], tid, rb[0]);
    __syncthreads();
    read_frags(0, 0);
    load_tile<AV, ATOT, NT, BK, VW>(xres, p.I, xrows, D * BK, klen, tid, ra[0]);
    load_tile<BV, BTOT, NT, BK, VW>(wres, p.I, wrows, D * BK, klen, tid, rb[0]);
    const int nround = klen > 0 ? (klen + D * BK - 1) / (D * BK) : 0;
    for (int r = 0; r < nround; ++r) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int nx = (j + 1) % D;
            store_tile<AV, ATOT, NT, BK, LDK, VW, RELU_X>(sA[nx & 1], tid, ra[nx]);
            store_tile<BV, BTOT, NT, BK, LDK, VW>(sB[nx & 1], tid, rb[nx]);
            mfma(j & 1, 0, H);
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
            read_frags(nx & 1, nx & 1);
            const int knext = (r * D + j + 1 + D) * BK;
            load_tile<AV, ATOT, NT, BK, VW>(xres, p.I, xrows, knext, klen, tid, ra[nx]);
            load_tile<BV, BTOT, NT, BK, VW>(wres, p.I, wrows, knext, klen, tid, rb[nx]);
            mfma(j & 1, H, BK / 2);
            __builtin_amdgcn_sched_barrier(0);
        }
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
int fill_fc_bias(const FcParams& prm, hipStream_t st) {
    const BiasFill fill = make_bias_fill(prm.y, prm.bias, prm.N, prm.O, 1);
    return launch_bias_fills(&fill, 1, st);
}

// Batches of at most 64 images (NB blocks of 32): each wave owns OB blocks of
// 32 output features and a run of the reduction, for every image, and feeds
// the matrix cores straight from its registers: lane (i, h) loads row i of
// the images' and of the weights' slab as float4s at taps 8q + 4h .. 8q + 4h
// + 3 of a 32-tap chunk, so its own registers hold the MFMA operands for
// every k-step (half h is the k index of the instruction) and no LDS stage
// or barrier sits in the reduction loop.  Two chunks are in flight per wave.
// The KW waves of a workgroup take consecutive runs of the reduction for the
// same outputs; their partial tiles are summed through LDS in a fixed order,
// and a split reduction (grid y > 1) adds the workgroups' sums atomically to
// an output pre-filled with the bias.  With a small batch the weight tiles
// are not shared between waves, so nothing is lost by skipping LDS, and the
// grid can be sized to two waves per SIMD however few output tiles there are
// (AlexNet's fc8 at batch 64 has 16 tiles of 64 x 64).
template <int NB, int OB, int KW, bool RELU_X>
__global__ void __launch_bounds__(64 * KW) fc_direct_f32(FcParams p) {
    constexpr int Q = 4;            // float4 loads per row and chunk (32 taps)
    constexpr int TILES = NB * OB;  // 32 x 32 accumulator tiles per wave
    __shared__ float red[KW * TILES * 16 * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i = lane & 31, h = lane >> 5;
    const int o0 = blockIdx.x * (OB * 32);
    const int kbase = (blockIdx.y * KW + wave) * p.kchunk;  // this wave's first tap
    const int kend = min(p.I, kbase + p.kchunk);
    const int nch = kend > kbase ? (kend - kbase + 31) / 32 : 0;
    // rows past N (images) or past O (features) lie past the resources' ends
    const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(p.x), (short)0, p.N * p.I * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(p.w + (size_t)o0 * p.I), (short)0, min(OB * 32, p.O - o0) * p.I * 4, 0x00020000);

    floatx16 acc[TILES];
#pragma unroll
    for (int t = 0; t < TILES; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[t][v] = 0.0f;
    f32x4 xa[2][NB][Q], wb[2][OB][Q];
    auto load = [&](int c, int s) {
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int k = kbase + c * 32 + 8 * q + 4 * h;
            const bool ok = k < kend;  // I is a multiple of 4: a float4 is all in or all out
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                xa[s][nb][q] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                    xres, ok ? ((nb * 32 + i) * p.I + k) * 4 : kOutOfRange, 0, 0));
#pragma unroll
            for (int ob = 0; ob < OB; ++ob)
                wb[s][ob][q] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                    wres, ok ? ((ob * 32 + i) * p.I + k) * 4 : kOutOfRange, 0, 0));
        }
    };
    auto compute = [&](int s) {
#pragma unroll
        for (int q = 0; q < Q; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    float a = xa[s][nb][q][e];
                    if constexpr (RELU_X) a = a > 0.0f ? a : 0.0f;
#pragma unroll
                    for (int ob = 0; ob < OB; ++ob)
                        acc[nb * OB + ob] =
                            __builtin_amdgcn_mfma_f32_32x32x2f32(a, wb[s][ob][q][e], acc[nb * OB + ob], 0, 0, 0);
                }
    };
    if (nch > 0) load(0, 0);
    for (int c = 0; c < nch; c += 2) {
        load(c + 1, 1);  // past the run: reads zeros, not multiplied
        compute(0);
        if (c + 2 < nch) load(c + 2, 0);
        if (c + 1 < nch) compute(1);
    }

    // the waves' partial tiles, summed in wave order (lanes on consecutive words)
#pragma unroll
    for (int t = 0; t < TILES; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[(wave * TILES * 16 + t * 16 + v) * 64 + lane] = acc[t][v];
    __syncthreads();
    constexpr int E = TILES * 16 * 64;
    const bool split = gridDim.y > 1;
    for (int e = threadIdx.x; e < E; e += 64 * KW) {
        float sum = red[e];
#pragma unroll
        for (int w = 1; w < KW; ++w) sum += red[w * E + e];
        const int t = e >> 10, v = (e >> 6) & 15, l = e & 63;
        const int n = (t / OB) * 32 + 8 * (v >> 2) + 4 * (l >> 5) + (v & 3);
        const int o = o0 + (t % OB) * 32 + (l & 31);
        if (n < p.N && o < p.O) {
            float* dst = p.y + (size_t)n * p.O + o;
            if (split) {
                atomicAdd(dst, sum);
            } else {
                if (p.bias) sum += p.bias[o];
                if (p.relu) sum = sum > 0.0f ? sum : 0.0f;
                *dst = sum;
            }
        }
    }
}

// Batches of at most kGemvMaxN images: a matrix-vector product per image on
// the vector ALUs, since a 32-row MFMA tile would be mostly empty.  A
// workgroup owns R consecutive output features (4, or 1 when there are fewer
// than 4096 of them, so that the launch still has ~1000 workgroups) and its
// four waves take a quarter of the reduction each.  A lane streams the weight
// rows with 128-bit loads (VEC; 32-bit otherwise), four steps in flight,
// multiplies them by the images' inputs (served from L2), and the partial
// sums are reduced across the wave and then through LDS across the four
// waves.  The bias and the ReLU are applied as the sum is stored: no split,
// no bias fill and no atomics, so the result is the same from run to run.
template <int N, int R, bool VEC, bool RELU_X>
__global__ void __launch_bounds__(256) fc_gemv_f32(FcParams p) {
    typedef typename std::conditional<VEC, float4, float>::type V;
    constexpr int W = VEC ? 4 : 1;                   // floats per load
    constexpr int U = 4;                             // steps in flight
    __shared__ float part[4][R][N];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int o0 = blockIdx.x * R;
    const int KV = p.I / W;                          // loads per row
    const int per = (KV + 3) / 4;                    // this wave's range
    const int kb = wave * per, ke = min(KV, kb + per);
    const V* wr[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        wr[r] = reinterpret_cast<const V*>(p.w + (size_t)min(o0 + r, p.O - 1) * p.I);
    const V* xr = reinterpret_cast<const V*>(p.x);
    auto dot = [](const V& a, const V& b) -> float {
        if constexpr (VEC) return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
        else return a * b;
    };
    auto relu_v = [](V v) -> V {
        if constexpr (!RELU_X) return v;
        else if constexpr (VEC) return make_float4(fmaxf(v.x, 0.0f), fmaxf(v.y, 0.0f), fmaxf(v.z, 0.0f), fmaxf(v.w, 0.0f));
        else return fmaxf(v, 0.0f);
    };
    float acc[R][N];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int n = 0; n < N; ++n) acc[r][n] = 0.0f;
    int k = kb + lane;
    for (; k + (U - 1) * 64 < ke; k += U * 64) {
        V wv[U][R], xv[U][N];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int r = 0; r < R; ++r) wv[u][r] = wr[r][k + u * 64];
#pragma unroll
            for (int n = 0; n < N; ++n) xv[u][n] = relu_v(xr[(size_t)n * KV + k + u * 64]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int n = 0; n < N; ++n) acc[r][n] += dot(wv[u][r], xv[u][n]);
    }
    for (; k < ke; k += 64) {
#pragma unroll
        for (int n = 0; n < N; ++n) {
            const V xv = relu_v(xr[(size_t)n * KV + k]);
#pragma unroll
            for (int r = 0; r < R; ++r) acc[r][n] += dot(wr[r][k], xv);
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int n = 0; n < N; ++n) {
            float v = acc[r][n];
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
            if (lane == 0) part[wave][r][n] = v;
        }
    __syncthreads();
    const int t = threadIdx.x;
    if (t < R * N) {
        const int r = t / N, n = t - r * N;
        const int o = o0 + r;
        if (o < p.O) {
            float v = (part[0][r][n] + part[1][r][n]) + (part[2][r][n] + part[3][r][n]);
            if (p.bias) v += p.bias[o];
            if (p.relu) v = v > 0.0f ? v : 0.0f;
            p.y[(size_t)n * p.O + o] = v;
        }
    }
}

template <int N, int R>
int launch_fc_gemv_r(const FcParams& prm, bool vec, bool relu_in, hipStream_t st) {
    const dim3 grid(ceil_div(prm.O, R)), block(256);
    if (vec) {
        if (relu_in) enqueue((fc_gemv_f32<N, R, true, true>), grid, block, 0, st, prm);
        else enqueue((fc_gemv_f32<N, R, true, false>), grid, block, 0, st, prm);
    } else {
        if (relu_in) enqueue((fc_gemv_f32<N, R, false, true>), grid, block, 0, st, prm);
        else enqueue((fc_gemv_f32<N, R, false, false>), grid, block, 0, st, prm);
    }
    return check_launch("fc_gemv_f32");
}

template <int N>
int launch_fc_gemv(const FcParams& prm, bool vec, bool relu_in, hipStream_t st) {
    return prm.O >= 4096 ? launch_fc_gemv_r<N, 4>(prm, vec, relu_in, st)
                         : launch_fc_gemv_r<N, 1>(prm, vec, relu_in, st);
}

// Several outputs at once (FillJobs).
__global__ void bias_fill_multi(FillJobsOf<kMaxBiasFills> f) { run_fills(f); }

// Tile and reduction split of an FC layer (one rule for launch_fc and the
// network planner).
struct FcGeom {
    int tm, tn, unit;  // workgroup tile, reduction granule of one split
    int target;        // workgroups to aim for (two to four per compute unit)
};

// tm: 32 (launch_fc_cfg<1, 4, 1, 1, 32, 4>) or 64 (launch_fc_cfg<2, 2, 1, 1, bk, 4>,
// bk 16 or 32); target in workgroups for a batch of N.
FcGeom fc_geom(int tm, int N, int bk = 16) {
    if (tm == 32) return FcGeom{32, 128, 4 * 32, 512};
    return FcGeom{64, 64, 4 * bk, N <= 64 ? 512 : 1024};
}

// Splits and the reduction length per split.
int fc_split(const FcGeom& g, int N, int I, int O, int* kchunk) {
    const int tiles = ceil_div(N, g.tm) * ceil_div(O, g.tn);
    // Enough splits to reach the target, with at least one ring round per
    // split; with 64-image tiles at least four, since there a layer with few
    // output tiles (AlexNet's fc8 at batch 64: 16) is bound by its atomic
    // partial sums rather than by its weight stream (fc8 18 -> 15 us).
    const int min_rounds = g.tm == 64 ? 4 : 1;
    int splits = std::min(ceil_div(g.target, tiles), std::max(1, I / (min_rounds * g.unit)));
    splits = std::max(splits, 1);
    *kchunk = ceil_div(ceil_div(I, splits), g.unit) * g.unit;
    return ceil_div(I, *kchunk);
}

// relu_left, prefilled: see launch_fc.
template <int WMW, int WNW, int FM, int FN, int BK, int D, bool VEC, bool RELU_X>
int launch_fc_cfg(const FcParams& prm0, const FcGeom& g, hipStream_t st, bool* relu_left, bool prefilled) {
    constexpr int TM = WMW * FM * 32;
    constexpr int TN = WNW * FN * 32;
    if (g.tm != TM || g.tn != TN || g.unit != D * BK)
        return fail(CNN_ERR_UNSUPPORTED, "fc: tile geometry out of step with fc_geom");
    FcParams prm = prm0;
    const int splits = fc_split(g, prm.N, prm.I, prm.O, &prm.kchunk);
    dim3 grid(ceil_div(prm.O, TN), ceil_div(prm.N, TM), splits);
    dim3 block(64 * WMW * WNW);
    if (splits > 1) {
        if (!prefilled) {
            const int rc = fill_fc_bias(prm, st);
            if (rc != CNN_OK) return rc;
        }
        enqueue((fc_gemm_f32<WMW, WNW, FM, FN, BK, D, VEC, true, RELU_X>), grid, block, 0, st, prm);
        int rc = check_launch("fc_gemm_f32");
        if (rc != CNN_OK) return rc;
        if (prm.relu && relu_left) {  // the caller applies it
            *relu_left = true;
            return CNN_OK;
        }
        if (prm.relu) return launch_relu(prm.y, prm.y, (int64_t)prm.N * prm.O, st);
        return CNN_OK;
    }
    enqueue((fc_gemm_f32<WMW, WNW, FM, FN, BK, D, VEC, false, RELU_X>), grid, block, 0, st, prm);
    return check_launch("fc_gemm_f32");
}

// Direct kernel: reduction run per wave, so that the grid has about
// kDirectWaves waves (two per SIMD) whatever the number of output blocks.
constexpr int kDirectWaves = 2048;
struct FcDirectGeom {
    int ob, kw;  // 32-feature blocks per wave, waves per workgroup
};
int fc_direct_split(const FcDirectGeom& g, int I, int O, int* kchunk) {
    const int groups = ceil_div(O, 32 * g.ob);
    const int per_group = std::max(1, kDirectWaves / groups);      // waves along the reduction
    *kchunk = std::max(32, ceil_div(ceil_div(I, per_group), 32) * 32);  // whole 32-tap chunks
    return ceil_div(ceil_div(I, *kchunk), g.kw);
}

template <int NB, int OB, int KW, bool RELU_X>
int launch_fc_direct_t(const FcParams& prm0, hipStream_t st, bool* relu_left, bool prefilled) {
    FcParams prm = prm0;
    const int splits = fc_direct_split(FcDirectGeom{OB, KW}, prm.I, prm.O, &prm.kchunk);
    const dim3 grid(ceil_div(prm.O, 32 * OB), splits), block(64 * KW);
    if (splits > 1 && !prefilled) {
        const int rc = fill_fc_bias(prm, st);
        if (rc != CNN_OK) return rc;
    }
    enqueue((fc_direct_f32<NB, OB, KW, RELU_X>), grid, block, 0, st, prm);
    int rc = check_launch("fc_direct_f32");
    if (rc != CNN_OK || splits == 1 || !prm.relu) return rc;
    if (relu_left) {  // the caller applies it
        *relu_left = true;
        return CNN_OK;
    }
    return launch_relu(prm.y, prm.y, (int64_t)prm.N * prm.O, st);
}

template <int OB, int KW>
int launch_fc_direct(const FcParams& prm, bool relu_in, hipStream_t st, bool* relu_left, bool prefilled) {
    if (prm.N <= 32)
        return relu_in ? launch_fc_direct_t<1, OB, KW, true>(prm, st, relu_left, prefilled)
                       : launch_fc_direct_t<1, OB, KW, false>(prm, st, relu_left, prefilled);
    return relu_in ? launch_fc_direct_t<2, OB, KW, true>(prm, st, relu_left, prefilled)
                   : launch_fc_direct_t<2, OB, KW, false>(prm, st, relu_left, prefilled);
}

// The configurations (cnn_fc_fwd_config).
struct FcConfig {
    const char* name;
    int max_n;      // largest batch it takes
    bool need_vec;  // 128-bit loads only (I % 4 == 0, 16-byte aligned x and w)
};
const FcConfig kFcConfigs[] = {
    {"tiled, 64 images x 64 features, 2x2 waves, 16-tap slabs", 1 << 30, false},
    {"tiled, 32 images x 128 features, 1x4 waves, 32-tap slabs", 1 << 30, false},
    {"direct, 32 features per wave, 8 waves", 64, true},
    {"matrix-vector", kGemvMaxN, false},
    {"tiled, 64 images x 64 features, 2x2 waves, 32-tap slabs", 1 << 30, false},
};
constexpr int kNumFcConfigs = sizeof(kFcConfigs) / sizeof(kFcConfigs[0]);

// Built-in choice (vec: 128-bit loads possible), from kernel-trace times of
// every configuration on the networks' FC shapes at batches 1 to 256 (`python
// bench.py --fc-config-table`).  Layers with few output features have few
// output tiles; the tiled kernels then split the reduction many ways (1M
// atomic partial sums for AlexNet's fc8 at batch 64) or, with a short
// reduction, hardly at all (LeNet's 500 -> 10 at batch 64: one
// workgroup, 13 us), while the direct kernel sizes its grid to two waves per
// SIMD whatever the number of tiles: at most 32 images it took fc8 (4096 ->
// 1000) at batch 16 from 8.4 to 6.0 us, and 500 -> 10 at batch 64 from 13.0
// to 5.4 us.  It reads the images once per 32 features, twice as often as
// the 64 x 64 tiles, which is what limits it on wide layers at batch 64
// (fc6 64.0 against 50.0 us).  In the network at batch 16, with the input's
// ReLU deferred from the layer before, fc7 (4096 -> 4096) took 21.4 us direct
// against 20.2 tiled.  Above 64 images, layers of at most 1024 features run
// 3-45% faster on the 32 x 128 tiles (twice the row tiles of 64 x 64).  At
// 33-64 images the wide layers take 32-tap slabs on the 64 x 64 tiles (the
// same split count, twice the matrix-core work per barrier): AlexNet's fc6
// at batch 64 went from 45 to 43 us in the network; fc8 keeps 16-tap slabs,
// whose finer split granule gives it twice the splits.
int fc_heuristic(int N, int I, int O, bool vec) {
    if (N <= kGemvMaxN) return 3;
    if (N > 32 && N <= 64 && O >= 2048 && I >= 4096) return 4;
    if (vec && N <= 64 && I <= 4096 && O <= (N <= 32 ? 2048 : 512)) return 2;
    if (N <= 32) return 1;
    if (N > 64 && O <= 1024 && I >= 256) return 1;
    return 0;
}

int fc_config_splits(int cfg, int N, int I, int O) {
    int kchunk;
    switch (cfg) {
        case 0: return fc_split(fc_geom(64, N), N, I, O, &kchunk);
        case 1: return fc_split(fc_geom(32, N), N, I, O, &kchunk);
        case 2: return fc_direct_split(FcDirectGeom{1, 8}, I, O, &kchunk);
        case 4: return fc_split(fc_geom(64, N, 32), N, I, O, &kchunk);
        default: return 1;
    }
}

}  // namespace

int fc_num_configs() { return kNumFcConfigs; }

const char* fc_config_name(int i) { return (i >= 0 && i < kNumFcConfigs) ? kFcConfigs[i].name : nullptr; }

int fc_splits(int N, int I, int O) {
    return N > 0 ? fc_config_splits(fc_heuristic(N, I, O, I % 4 == 0), N, I, O) : 1;
}

int launch_bias_fills(const BiasFill* jobs, int n, hipStream_t st) {
    for (int j0 = 0; j0 < n; j0 += kMaxBiasFills) {
        FillJobsOf<kMaxBiasFills> f;
        f.n = std::min(kMaxBiasFills, n - j0);
        int64_t most = 0;
        for (int j = 0; j < f.n; ++j) {
            f.job[j] = jobs[j0 + j];
            most = std::max(most, (int64_t)f.job[j].total);
        }
        if (most == 0) continue;
        enqueue(bias_fill_multi, dim3((unsigned)std::min<int64_t>(ceil_div64(most, 256), 2048)),
                           dim3(256), 0, st, f);
        const int rc = check_launch("bias_fill_multi");
        if (rc != CNN_OK) return rc;
    }
    return CNN_OK;
}

int launch_fc(const float* x, int N, int I, const float* w, const float* bias, int O, int relu,
              float* y, hipStream_t st, bool relu_in, bool* relu_left, bool prefilled, int config) {
    if (relu_left) *relu_left = false;
    if (config < -1 || config >= kNumFcConfigs) return fail(CNN_ERR_INVALID, "fc: no configuration %d", config);
    if (N == 0) return CNN_OK;
    // buffer offsets within a workgroup's rows are 31-bit
    if ((int64_t)128 * I * 4 >= ((int64_t)1 << 31))
        return fail(CNN_ERR_UNSUPPORTED, "fc: %d input features exceed this kernel's 2^22 limit", I);
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
    int cfg = config;
    if (cfg < 0) {
        cfg = fc_heuristic(N, I, O, vec);
        if (kFcConfigs[cfg].need_vec && !vec) cfg = N <= 32 ? 1 : 0;
    }
    if (N > kFcConfigs[cfg].max_n)
        return fail(CNN_ERR_UNSUPPORTED, "fc: configuration %d takes at most %d images", cfg, kFcConfigs[cfg].max_n);
    if (kFcConfigs[cfg].need_vec && !vec)
        return fail(CNN_ERR_UNSUPPORTED, "fc: configuration %d needs I %% 4 == 0 and 16-byte aligned x and w", cfg);
#define CNN_FC_CFG(G, WMW, WNW, FM, FN, BK, D)                                                                     \
    (vec ? (relu_in ? launch_fc_cfg<WMW, WNW, FM, FN, BK, D, true, true>(prm, G, st, relu_left, prefilled)          \
                    : launch_fc_cfg<WMW, WNW, FM, FN, BK, D, true, false>(prm, G, st, relu_left, prefilled))        \
         : (relu_in ? launch_fc_cfg<WMW, WNW, FM, FN, BK, D, false, true>(prm, G, st, relu_left, prefilled)         \
                    : launch_fc_cfg<WMW, WNW, FM, FN, BK, D, false, false>(prm, G, st, relu_left, prefilled)))
    switch (cfg) {
        case 0: return CNN_FC_CFG(fc_geom(64, N), 2, 2, 1, 1, 16, 4);  // 64 x 64
        case 1: return CNN_FC_CFG(fc_geom(32, N), 1, 4, 1, 1, 32, 4);  // 32 images x 128 features
        case 2: return launch_fc_direct<1, 8>(prm, relu_in, st, relu_left, prefilled);
        case 4: return CNN_FC_CFG(fc_geom(64, N, 32), 2, 2, 1, 1, 32, 4);  // 64 x 64, 32-tap slabs
        default:
            static_assert(kGemvMaxN == 2, "one instantiation per batch size");
            return N == 1 ? launch_fc_gemv<1>(prm, vec, relu_in, st) : launch_fc_gemv<2>(prm, vec, relu_in, st);
    }
#undef CNN_FC_CFG
}

}  // namespace cnn
