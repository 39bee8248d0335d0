// Dense layer of the synthetic MLP denoiser on fp32 MFMA: one block per output
// tile (the tile itself is computed in linear_tile.h).  At the policy
// network's sizes (100 rows in a window, one in the sequential chain) the
// layer is bound by latency and by the cost of dispatching waves, not by the
// matrix core: few waves with a few dozen MFMAs each beat many waves with a
// handful.
#include "linear_tile.h"

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

}  // namespace pd
