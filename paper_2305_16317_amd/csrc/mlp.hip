// Dense layer y = act(x W^T + bias) (or + shift[n_row] for the first layer,
// which carries b1 + e_n) of the synthetic MLP denoiser, on fp32 MFMA.
//
// v_mfma_f32_16x16x4f32 operand layout (wave64): A[i][k] sits in lane
// i + 16 k, B[k][j] in lane j + 16 k, and D[i][j] in lane j + 16 (i / 4),
// register i % 4.  Each lane loads four consecutive k of its row of x and of
// W as one float4; step q of the four MFMAs then pairs element q of both
// vectors, i.e. lane group h = lane / 16 covers k = k0 + 4 h + q.  Any
// permutation of k works as long as A and B agree, so the loads stay
// contiguous.
//
// One block = one 16 x 16 output tile; its 16 waves take every 16th chunk of
// 16 k and the partial tiles are summed through LDS in a fixed order.  At the
// policy network's sizes (100 rows in a window, one in the sequential chain)
// the layer is bound by latency, not by the matrix core: more waves per tile
// put more loads in flight (16 waves: the sequential chain 3.3 -> 2.2 ms).
#include "pd_internal.h"

namespace pd {
namespace {

constexpr int kLinWaves = 16;   // waves per block, splitting K

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float gelu_exact(float u) {
    return 0.5f * u * (1.0f + erff(u / 1.41421356237f));
}

template <bool GATHER>
__global__ __launch_bounds__(kLinWaves * 64) void k_linear(LinearArgs a, const float* __restrict__ xd,
                                                RowSrc src, int64_t D, float* __restrict__ y) {
    const int groups = src.active ? *src.active : src.max_groups;
    const int M = groups * src.group;
    const int m0 = blockIdx.y * 16, n0 = blockIdx.x * 16;
    if (m0 >= M) return;
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
    const int nr = min(n0 + li, N - 1);
    const float* wrow = a.W + (int64_t)nr * K;

    // the epilogue's bias (or per-timestep shift) of this lane's four outputs,
    // fetched before the reduction so its latency hides behind the MFMAs
    const int n_out = min(n0 + li, N - 1);
    float addv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int m = min(m0 + 4 * h + q, M - 1);
        addv[q] = a.shift != nullptr ? a.shift[(int64_t)src.n[m / src.group] * N + n_out]
                                     : a.bias[n_out];
    }

    // this wave's chunks are c = w, w + 4, ...; kBatch of them are loaded
    // before any is multiplied, so their loads are in flight together
    constexpr int kBatch = 4;
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    const int nchunks = (K + 15) / 16;
    for (int c0 = w; c0 < nchunks; c0 += kLinWaves * kBatch) {
        f4 av[kBatch], bv[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int k = (c0 + kLinWaves * u) * 16 + 4 * h;
            const bool ok = c0 + kLinWaves * u < nchunks && k < K;   // K is a multiple of 4
            const int kk = ok ? k : 0;
            const f4 xa = *reinterpret_cast<const f4*>(xrow + kk);
            const f4 wb = *reinterpret_cast<const f4*>(wrow + kk);
            av[u] = ok ? xa : f4{0.f, 0.f, 0.f, 0.f};
            bv[u] = ok ? wb : f4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u][q], bv[u][q], acc, 0, 0, 0);
    }

    __shared__ f4 s_acc[kLinWaves][64];
    s_acc[w][lane] = acc;
    __syncthreads();
    if (w != 0) return;
    f4 sum = s_acc[0][lane];
#pragma unroll
    for (int v = 1; v < kLinWaves; ++v) sum += s_acc[v][lane];

    // D[i][j]: row m0 + 4 h + q, column n0 + li
    const int n = n0 + li;
    if (n >= N) return;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int m = m0 + 4 * h + q;
        if (m >= M) continue;
        float v = sum[q] + addv[q];
        if (a.act == ACT_GELU) v = gelu_exact(v);
        y[(int64_t)m * N + n] = v;
    }
}

template <bool GATHER>
void launch(const LinearArgs& a, const float* xd, const RowSrc& src, int64_t D, float* y,
            hipStream_t s) {
    const int64_t Mmax = (int64_t)src.max_groups * src.group;
    if (Mmax == 0) return;
    if ((a.K % 4) != 0 || (GATHER && (D % 4) != 0))
        fail(PD_ERR_UNSUPPORTED, "mlp layer sizes must be multiples of 4");
    const dim3 grid((unsigned)((a.N + 15) / 16), (unsigned)((Mmax + 15) / 16));
    hipLaunchKernelGGL(k_linear<GATHER>, grid, dim3(kLinWaves * 64), 0, s, a, xd, src, D, y);
    PD_HIP(hipGetLastError());
}

}  // namespace

void launch_linear_gather(const LinearArgs& a, const RowSrc& src, int64_t D, float* y,
                          hipStream_t s) {
    launch<true>(a, nullptr, src, D, y, s);
}

void launch_linear_dense(const LinearArgs& a, const float* x, const RowSrc& rows, float* y,
                         hipStream_t s) {
    launch<false>(a, x, rows, 0, y, s);
}

}  // namespace pd
