// Exact epsilon of an equal-weight isotropic 2-D Gaussian mixture noised by
// the training schedule: eps = coef_n (x - a_n sum_k w_k mu_k) with
// w = softmax_k(-|x - a_n mu_k|^2 / (2 s_n^2)).  One thread per row; the
// per-timestep constants are float tables built in double on the host.
#include "pd_internal.h"

namespace pd {
namespace {

constexpr int kMaxK = 64;

__global__ __launch_bounds__(256) void k_gmm_eps(GmmParams g, RowSrc src,
                                                 float* __restrict__ eps) {
    const int groups = src.active ? *src.active : src.max_groups;
    const int64_t rows = (int64_t)groups * src.group;
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    const int gi = (int)(r / src.group), b = (int)(r % src.group);
    const int64_t sl = src.slot ? src.slot[gi] : gi;
    const float* x = src.base + sl * src.slot_stride + (int64_t)b * 2;
    const int n = src.n[gi];
    const float x0 = x[0], x1 = x[1];
    const float a = g.a[n], inv2s2 = g.inv2s2[n], coef = g.coef[n];
    // two passes over the components (max, then weights) keep no per-k array
    auto logit = [&](int k) {
        const float d0 = x0 - a * g.means[2 * k];
        const float d1 = x1 - a * g.means[2 * k + 1];
        return -(d0 * d0 + d1 * d1) * inv2s2;
    };
    float mx = -INFINITY;
    for (int k = 0; k < g.K; ++k) mx = fmaxf(mx, logit(k));
    float sw = 0.f, m0 = 0.f, m1 = 0.f;
    for (int k = 0; k < g.K; ++k) {
        const float w = expf(logit(k) - mx);
        sw += w;
        m0 += w * g.means[2 * k];
        m1 += w * g.means[2 * k + 1];
    }
    m0 = m0 / sw;
    m1 = m1 / sw;
    float* o = eps + r * 2;
    o[0] = coef * (x0 - a * m0);
    o[1] = coef * (x1 - a * m1);
}

}  // namespace

void launch_gmm_eps(const GmmParams& g, const RowSrc& src, float* eps, hipStream_t s) {
    if (g.K > kMaxK) fail(PD_ERR_UNSUPPORTED, "gmm2d supports at most 64 components");
    const int64_t rows = (int64_t)src.max_groups * src.group;
    if (rows == 0) return;
    hipLaunchKernelGGL(k_gmm_eps, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, g, src,
                       eps);
    PD_HIP(hipGetLastError());
}

}  // namespace pd
