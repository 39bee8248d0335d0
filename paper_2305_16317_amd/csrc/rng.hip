// Up-front noise of Algorithm 1 (prior point and the noise of every step)
// from the counter-based draws of philox.h: one thread turns one 128-bit
// counter block into four normals.
#include "pd_internal.h"
#include "philox.h"

namespace pd {
namespace {

// Values 4q .. 4q + 3 of counter stream rng_stream (those below count) into out.
__device__ __forceinline__ void normals_quad(uint64_t seed, uint32_t rng_stream, int64_t q,
                                             int64_t count, const float* __restrict__ scale,
                                             int64_t per_scale, float* __restrict__ out) {
    float v[4];
    normals4(seed, rng_stream, q, v);
    const int64_t base = 4 * q;
    if (scale != nullptr) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (base + e < count) v[e] = scale[(base + e) / per_scale] * v[e];
    }
    if (base + 3 < count && (count & 3) == 0) {
        *reinterpret_cast<float4*>(out + base) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (base + e < count) out[base + e] = v[e];
    }
}

__global__ __launch_bounds__(256) void k_normals(uint64_t seed, uint32_t rng_stream,
                                                 int64_t count, const float* __restrict__ scale,
                                                 int64_t per_scale, float* __restrict__ out) {
    const int64_t nq = (count + 3) / 4;
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nq; q += step)
        normals_quad(seed, rng_stream, q, count, scale, per_scale, out);
}

// The prior (stream 0, BD values into x0) and then the noise (stream 1,
// noise_count values) share one grid of quads; the first block also starts
// the Picard loop when has_init is set.
__global__ __launch_bounds__(256) void k_sample_setup(uint64_t seed, int64_t BD, float* __restrict__ x0,
                                                      int64_t noise_count, const float* __restrict__ scale,
                                                      int64_t per_scale, float* __restrict__ noise,
                                                      PicardInit init, int has_init) {
    if (has_init && blockIdx.x == 0) picard_init_body(init);
    const int64_t nq0 = (BD + 3) / 4, nq = nq0 + (noise_count + 3) / 4;
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nq; q += step) {
        if (q < nq0) normals_quad(seed, 0, q, BD, nullptr, 1, x0);
        else normals_quad(seed, 1, q - nq0, noise_count, scale, per_scale, noise);
    }
}

}  // namespace

void launch_normals(uint64_t seed, uint32_t rng_stream, int64_t count, const float* scale,
                    int64_t per_scale, float* out, hipStream_t s) {
    if (count <= 0) return;
    const int64_t nq = (count + 3) / 4;
    int64_t blocks = (nq + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_normals, dim3((unsigned)blocks), dim3(256), 0, s, seed, rng_stream,
                       count, scale, per_scale, out);
    PD_HIP(hipGetLastError());
}

void launch_sample_setup(uint64_t seed, int64_t BD, float* x0, int64_t noise_count,
                         const float* scale, int64_t per_scale, float* noise,
                         const PicardInit* init, hipStream_t s) {
    if (!noise) noise_count = 0;
    const int64_t nq = (BD + 3) / 4 + (noise_count + 3) / 4;
    int64_t blocks = (nq + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    const PicardInit none{};
    hipLaunchKernelGGL(k_sample_setup, dim3((unsigned)blocks), dim3(256), 0, s, seed, BD, x0,
                       noise_count, scale, per_scale, noise, init ? *init : none, init ? 1 : 0);
    PD_HIP(hipGetLastError());
}

}  // namespace pd
