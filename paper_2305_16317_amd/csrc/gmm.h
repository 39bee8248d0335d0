// The mixture's one-workgroup Picard loop, drawing its own prior and noise.
#pragma once

#include "pd_internal.h"

namespace pd {

// The up-front draws of a sample (Algorithm 1's setup) made inside the loop's
// workgroup instead of by a separate launch: the prior x_0 is values 0 .. BD-1
// of counter stream 0 and the noise of step i is values i BD .. i BD + BD - 1
// of stream 1 times zstd[i] (philox.h), so both are those of launch_normals and
// launch_sample_setup with the same seed.
struct GmmDraw {
    int32_t on;            // 0: read a.x0 and a.noise as given
    uint64_t seed;
    const float* zstd;     // [T] noise standard deviation per step, or nullptr (no noise)
};

// Whether the loop keeps every step's noise in LDS (what drawing in the loop
// needs) for these sizes within max_lds bytes.
bool gmm_loop_stages_noise(int T, int K, int p, int batch, size_t max_lds);
// The loop of launch_gmm_picard_loop; with draw.on it draws x_0 and the noise
// itself (gmm_loop_stages_noise must hold) and reads neither a.x0 nor a.noise.
void launch_gmm_picard_loop(const GmmLoopArgs& a, const GmmDraw& draw, size_t max_lds,
                            hipStream_t s);

}  // namespace pd
