// Counter-based normal draws shared by the kernels that draw the up-front
// noise of Algorithm 1 (the prior point and every step's noise): Philox4x32-10
// (Salmon, Moraes, Dror, Shaw, SC'11) with Box-Muller in double precision.
// Counter block q of stream s is (q mod 2^32, q / 2^32, s, 0) under the key
// (seed mod 2^32, seed / 2^32); it gives values 4q .. 4q + 3 of the stream.
#pragma once

#include <cstdint>

namespace pd {

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

// Values 4q .. 4q + 3 of counter stream rng_stream, rounded to float.
__device__ __forceinline__ void normals4(uint64_t seed, uint32_t rng_stream, int64_t q, float (&v)[4]) {
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
    v[0] = (float)(r01 * co1);
    v[1] = (float)(r01 * s1);
    v[2] = (float)(r23 * co3);
    v[3] = (float)(r23 * s3);
}

}  // namespace pd
