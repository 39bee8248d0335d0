// One output tile of a dense layer y = act(x W^T + bias) (or + shift[n_row]
// for the first layer, which carries b1 + e_n) of the synthetic MLP denoiser,
// on fp32 MFMA.  Shared by the layer kernel (mlp.hip) and the fused last
// layer and Picard update (picard.hip), so both compute bitwise the same
// epsilon.
//
// v_mfma_f32_16x16x4f32 operand layout (wave64): A[i][k] sits in lane
// i + 16 k, B[k][j] in lane j + 16 k, and D[i][j] in lane j + 16 (i / 4),
// register i % 4.  Each lane loads four consecutive k of its row of x and of
// W as one float4; step q of the four MFMAs then pairs element q of both
// vectors, i.e. lane group h = lane / 16 covers k = k0 + 4 h + q.  Any
// permutation of k works as long as A and B agree, so the loads stay
// contiguous.
//
// A tile is 16 rows x (16 kNSub) columns.  The block's kLinWaves waves split
// K into contiguous runs of 16-wide chunks; each wave multiplies its x chunk
// against kNSub column groups of W (the x operand is loaded once for all of
// them), and the partial tiles are summed through LDS in wave order.
#pragma once

#include "pd_internal.h"

namespace pd {

#ifndef PD_LIN_WAVES
#define PD_LIN_WAVES 8
#endif
#ifndef PD_LIN_NSUB
#define PD_LIN_NSUB 1
#endif
constexpr int kLinWaves = PD_LIN_WAVES;   // waves per block, splitting K
constexpr int kNSub = PD_LIN_NSUB;        // 16-column groups per block
constexpr int kLinBatch = 8;              // chunks whose loads are in flight together
static_assert(kLinWaves * 64 >= 256 * kNSub, "every output of the tile needs a thread");

__device__ __forceinline__ float gelu_exact(float u) {
    return 0.5f * u * (1.0f + erff(u / 1.41421356237f));
}

// Rows of the layer's input: gathered from the window's ring slots (GATHER,
// the first layer) or a dense [M][K] buffer.  M rows are valid; the tile
// starts at row m0 < M and column n0.  Every thread of the block calls it.
template <bool GATHER>
__device__ __forceinline__ void linear_tile(const LinearArgs& a, const float* __restrict__ xd,
                                            const RowSrc& src, int64_t D, float* __restrict__ y,
                                            int M, int m0, int n0) {
    typedef float f4 __attribute__((ext_vector_type(4)));
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int li = lane & 15, h = lane >> 4;
    const int K = a.K, N = a.N;

    // row pointer of this lane's A row (clamped rows are computed, not stored)
    const int mr = min(m0 + li, M - 1);
    const float* xrow;
    if (GATHER) {
        const int g = mr / src.group, b = mr % src.group;
        const int64_t sl = src.slot ? src.slot[g] : g;
        xrow = src.base + sl * src.slot_stride + (int64_t)b * D;
    } else {
        xrow = xd + (int64_t)mr * K;
    }
    const float* wrow[kNSub];
#pragma unroll
    for (int s = 0; s < kNSub; ++s) wrow[s] = a.W + (int64_t)min(n0 + 16 * s + li, N - 1) * K;

    // epilogue: thread tid owns output (row m0 + 4 (l / 16) + q, column
    // n0 + 16 s + l % 16) with l = tid % 64, q = (tid / 64) % 4, s = tid / 256
    // (threads past 64 * 4 * kNSub own none); its bias or per-timestep shift
    // is fetched before the products so the latency hides behind them
    const int el = threadIdx.x & 63, eq = (threadIdx.x >> 6) & 3, es = threadIdx.x >> 8;
    const bool owner = es < kNSub;
    const int em = m0 + 4 * (el >> 4) + eq, en = n0 + 16 * es + (el & 15);
    float addv = 0.f;
    if (owner) {
        const int mc = min(em, M - 1), nc = min(en, N - 1);
        addv = a.shift != nullptr ? a.shift[(int64_t)row_timestep(src, mc / src.group) * N + nc] : a.bias[nc];
    }

    // this wave's chunks: a contiguous run of 16-wide k chunks
    const int nchunks = (K + 15) / 16;
    const int per = (nchunks + kLinWaves - 1) / kLinWaves;
    const int c_begin = w * per, c_end = min(c_begin + per, nchunks);
    f4 acc[kNSub];
#pragma unroll
    for (int s = 0; s < kNSub; ++s) acc[s] = f4{0.f, 0.f, 0.f, 0.f};
    for (int c0 = c_begin; c0 < c_end; c0 += kLinBatch) {
        f4 av[kLinBatch], bv[kLinBatch][kNSub];
#pragma unroll
        for (int u = 0; u < kLinBatch; ++u) {
            const int k = (c0 + u) * 16 + 4 * h;
            const bool ok = c0 + u < c_end && k < K;   // K is a multiple of 4
            const int kk = ok ? k : 0;
            const f4 xa = *reinterpret_cast<const f4*>(xrow + kk);
            av[u] = ok ? xa : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < kNSub; ++s) {
                const f4 wb = *reinterpret_cast<const f4*>(wrow[s] + kk);
                bv[u][s] = ok ? wb : f4{0.f, 0.f, 0.f, 0.f};
            }
        }
#pragma unroll
        for (int u = 0; u < kLinBatch; ++u)
#pragma unroll
            for (int s = 0; s < kNSub; ++s)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    acc[s] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u][q], bv[u][s][q], acc[s], 0, 0, 0);
    }

    // partial tiles, [wave][column group][register][lane]: conflict-free
    // writes (one register of 64 lanes at a time) and reads (64 lanes)
    __shared__ float s_acc[kLinWaves][kNSub][4][64];
#pragma unroll
    for (int s = 0; s < kNSub; ++s)
#pragma unroll
        for (int q = 0; q < 4; ++q) s_acc[w][s][q][lane] = acc[s][q];
    __syncthreads();
    if (owner && em < M && en < N) {
        float sum = s_acc[0][es][eq][el];
#pragma unroll
        for (int v = 1; v < kLinWaves; ++v) sum += s_acc[v][es][eq][el];
        float v = sum + addv;
        if (a.act == ACT_GELU) v = gelu_exact(v);
        y[(int64_t)em * N + en] = v;
    }
}

}  // namespace pd
