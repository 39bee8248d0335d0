// Dense layer of the synthetic MLP denoiser on fp32 MFMA: one block per output
// tile (the tile itself is computed in linear_tile.h).  At the policy
// network's sizes (100 rows in a window, one in the sequential chain) the
// layer is bound by latency and by the cost of dispatching waves, not by the
// matrix core: few waves with a few dozen MFMAs each beat many waves with a
// handful.
#include "linear_tile.h"
#include "mlp.h"

namespace pd {
namespace {

template <bool GATHER>
__global__ __launch_bounds__(kLinWaves * 64) void k_linear(LinearArgs a, const float* __restrict__ xd,
                                                RowSrc src, int64_t D, float* __restrict__ y) {
    const int groups = src.active ? *src.active : src.max_groups;
    const int M = groups * src.group;
    const int m0 = blockIdx.y * 16, n0 = blockIdx.x * (16 * kNSub);
    if (m0 >= M) return;
    linear_tile<GATHER>(a, xd, src, D, y, M, m0, n0);
}

// The last layer, then Heun's Euler prediction of each output the block
// wrote: the thread that stored an output (the tile's epilogue mapping) reads
// it back, so it sees its own store, and adds the drift
// A_m x + B_m eps with two rounded products and a rounded sum, as the scan's
// drift does.
__global__ __launch_bounds__(kLinWaves * 64) void k_linear_predict(LinearArgs a,
                                                                   const float* __restrict__ xd,
                                                                   RowSrc src, HeunPredictArgs h,
                                                                   float* y) {
    const int groups = src.active ? *src.active : src.max_groups;
    const int M = groups * src.group;
    const int m0 = blockIdx.y * 16, n0 = blockIdx.x * (16 * kNSub);
    if (m0 >= M) return;
    linear_tile<false>(a, xd, src, 0, y, M, m0, n0);
    const int el = threadIdx.x & 63, eq = (threadIdx.x >> 6) & 3, es = threadIdx.x >> 8;
    const int em = m0 + 4 * (el >> 4) + eq, en = n0 + 16 * es + (el & 15);
    if (es < kNSub && em < M && en < a.N) {
        const LoopState cur = *h.st;
        const int j = em / src.group, b = em % src.group;
        const int m = cur.t + j;
        const int64_t BD = (int64_t)src.group * a.N;
        const int64_t c = (int64_t)b * a.N + en;
        const float x = h.ring[(int64_t)((m <= cur.f ? m : cur.f) % h.ring_slots) * BD + c];
        const float e = y[(int64_t)em * a.N + en];
        const float dr = __fadd_rn(__fmul_rn(h.A[m], x), __fmul_rn(h.B[m], e));
        h.xt[(int64_t)j * BD + c] = __fadd_rn(x, dr);
    }
}

template <bool GATHER>
void launch(const LinearArgs& a, const float* xd, const RowSrc& src, int64_t D, float* y,
            hipStream_t s) {
    const int64_t Mmax = (int64_t)src.max_groups * src.group;
    if (Mmax == 0) return;
    if ((a.K % 4) != 0 || (GATHER && (D % 4) != 0))
        fail(PD_ERR_UNSUPPORTED, "mlp layer sizes must be multiples of 4");
    const dim3 grid((unsigned)((a.N + 16 * kNSub - 1) / (16 * kNSub)), (unsigned)((Mmax + 15) / 16));
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

void launch_linear_dense_predict(const LinearArgs& a, const float* x, const RowSrc& rows,
                                 const HeunPredictArgs& h, float* y, hipStream_t s) {
    const int64_t Mmax = (int64_t)rows.max_groups * rows.group;
    if (Mmax == 0) return;
    if ((a.K % 4) != 0) fail(PD_ERR_UNSUPPORTED, "mlp layer sizes must be multiples of 4");
    const dim3 grid((unsigned)((a.N + 16 * kNSub - 1) / (16 * kNSub)), (unsigned)((Mmax + 15) / 16));
    hipLaunchKernelGGL(k_linear_predict, grid, dim3(kLinWaves * 64), 0, s, a, x, rows, h, y);
    PD_HIP(hipGetLastError());
}

}  // namespace pd
