// Up-front noise of Algorithm 1 (prior point and the noise of every step):
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) with Box-Muller in double
// precision.  One thread turns one 128-bit counter block into four normals.
#include "pd_internal.h"

namespace pd {
namespace {

constexpr uint32_t kPhiloxM0 = 0xD2511F53u;
constexpr uint32_t kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u;
constexpr uint32_t kPhiloxW1 = 0xBB67AE85u;

__device__ __forceinline__ void philox4x32_10(uint32_t& c0, uint32_t& c1, uint32_t& c2,
                                              uint32_t& c3, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += kPhiloxW0;
            k1 += kPhiloxW1;
        }
        const uint32_t lo0 = kPhiloxM0 * c0, hi0 = __umulhi(kPhiloxM0, c0);
        const uint32_t lo1 = kPhiloxM1 * c2, hi1 = __umulhi(kPhiloxM1, c2);
        const uint32_t n0 = hi1 ^ c1 ^ k0;
        const uint32_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
}

// Values 4q .. 4q + 3 of counter stream rng_stream (those below count) into out.
__device__ __forceinline__ void normals_quad(uint64_t seed, uint32_t rng_stream, int64_t q,
                                             int64_t count, const float* __restrict__ scale,
                                             int64_t per_scale, float* __restrict__ out) {
    const double kTwoPi = 6.283185307179586;   // 2 * pi in double
    const double kInv32 = 2.3283064365386963e-10;   // 2^-32
    uint32_t c0 = (uint32_t)q, c1 = (uint32_t)((uint64_t)q >> 32), c2 = rng_stream, c3 = 0;
    philox4x32_10(c0, c1, c2, c3, (uint32_t)seed, (uint32_t)(seed >> 32));
    const double u0 = ((double)c0 + 0.5) * kInv32;
    const double u1 = ((double)c1 + 0.5) * kInv32;
    const double u2 = ((double)c2 + 0.5) * kInv32;
    const double u3 = ((double)c3 + 0.5) * kInv32;
    const double r01 = sqrt(-2.0 * log(u0));
    const double r23 = sqrt(-2.0 * log(u2));
    double s1, co1, s3, co3;
    sincos(kTwoPi * u1, &s1, &co1);
    sincos(kTwoPi * u3, &s3, &co3);
    float v[4] = {(float)(r01 * co1), (float)(r01 * s1), (float)(r23 * co3), (float)(r23 * s3)};
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
