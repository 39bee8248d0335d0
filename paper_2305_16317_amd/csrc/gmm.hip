// Exact epsilon of an equal-weight isotropic 2-D Gaussian mixture noised by
// the training schedule: eps = coef_n (x - a_n sum_k w_k mu_k) with
// w = softmax_k(-|x - a_n mu_k|^2 / (2 s_n^2)).  One thread per row; the
// per-timestep constants are float tables built in double on the host.
// For this model the whole sampling loop (Picard or sequential) also runs in
// a single workgroup: the state is a few KB and fits in LDS.
#include "gmm.h"
#include "pd_internal.h"
#include "philox.h"

namespace pd {
namespace {

constexpr int kMaxK = 64;
constexpr size_t kLoopLdsMax = 64 * 1024;  // LDS of the single-workgroup loops

// Component means, read from memory (any K) or held in registers (K <= KM;
// the loops over components are then unrolled and the loads leave the loop).
struct MeansMem {
    static constexpr int kBound = 0;
    const float* p;
    __device__ float operator[](int i) const { return p[i]; }
};
template <int KM>
struct MeansReg {
    static constexpr int kBound = KM;
    float v[2 * KM];
    __device__ void load(const float* src, int K) {
#pragma unroll
        for (int i = 0; i < 2 * KM; ++i) v[i] = i < 2 * K ? src[i] : 0.f;
    }
    __device__ float operator[](int i) const { return v[i]; }
};

template <class M, class F>
__device__ __forceinline__ void for_components(int K, F&& f) {
    if constexpr (M::kBound > 0) {
#pragma unroll
        for (int k = 0; k < M::kBound; ++k)
            if (k < K) f(k);
    } else {
        for (int k = 0; k < K; ++k) f(k);
    }
}

// eps of one point from the constants of its network timestep n:
// a = sqrt(abar_n), inv2s2 = 1 / (2 s_n^2), coef = sqrt(1 - abar_n) / s_n^2.
template <class M>
__device__ __forceinline__ void gmm_eps_core(const M& means, int K, float a, float inv2s2,
                                             float coef, float x0, float x1, float& e0,
                                             float& e1) {
    // two passes over the components (max, then weights) keep no per-k array
    auto logit = [&](int k) {
        const float d0 = x0 - a * means[2 * k];
        const float d1 = x1 - a * means[2 * k + 1];
        return -(d0 * d0 + d1 * d1) * inv2s2;
    };
    float mx = -INFINITY;
    for_components<M>(K, [&](int k) { mx = fmaxf(mx, logit(k)); });
    float sw = 0.f, m0 = 0.f, m1 = 0.f;
    for_components<M>(K, [&](int k) {
        const float w = expf(logit(k) - mx);
        sw += w;
        m0 += w * means[2 * k];
        m1 += w * means[2 * k + 1];
    });
    m0 = m0 / sw;
    m1 = m1 / sw;
    e0 = coef * (x0 - a * m0);
    e1 = coef * (x1 - a * m1);
}

// The same eps with the components shared out over the four lanes of a quad
// (lane q takes components q, q + 4, ..., the means read from LDS): the
// largest logit and the three weighted sums are combined across the quad by
// two exchange steps (lanes l ^ 1, then l ^ 2).  Each step adds a lane's value
// to its partner's, and addition is commutative, so every lane of the quad
// ends with the same sums and the same eps.  All four lanes must be active.
template <int CTRL>
__device__ __forceinline__ float quad_partner(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xf,
                                                              0xf, false));
}
__device__ __forceinline__ void gmm_eps_quad(const float* means, int K, int q, float a,
                                             float inv2s2, float coef, float x0, float x1,
                                             float& e0, float& e1) {
    auto logit = [&](int k) {
        const float d0 = x0 - a * means[2 * k];
        const float d1 = x1 - a * means[2 * k + 1];
        return -(d0 * d0 + d1 * d1) * inv2s2;
    };
    float mx = -INFINITY;
    for (int k = q; k < K; k += 4) mx = fmaxf(mx, logit(k));
    mx = fmaxf(mx, quad_partner<0xb1>(mx));   // quad_perm [1, 0, 3, 2]
    mx = fmaxf(mx, quad_partner<0x4e>(mx));   // quad_perm [2, 3, 0, 1]
    float sw = 0.f, m0 = 0.f, m1 = 0.f;
    for (int k = q; k < K; k += 4) {
        const float w = expf(logit(k) - mx);
        sw += w;
        m0 += w * means[2 * k];
        m1 += w * means[2 * k + 1];
    }
    sw += quad_partner<0xb1>(sw);
    m0 += quad_partner<0xb1>(m0);
    m1 += quad_partner<0xb1>(m1);
    sw += quad_partner<0x4e>(sw);
    m0 += quad_partner<0x4e>(m0);
    m1 += quad_partner<0x4e>(m1);
    m0 = m0 / sw;
    m1 = m1 / sw;
    e0 = coef * (x0 - a * m0);
    e1 = coef * (x1 - a * m1);
}

__device__ __forceinline__ void gmm_eps_row(const GmmParams& g, int n, float x0, float x1,
                                            float& e0, float& e1) {
    gmm_eps_core(MeansMem{g.means}, g.K, g.a[n], g.inv2s2[n], g.coef[n], x0, x1, e0, e1);
}

__global__ __launch_bounds__(256) void k_gmm_eps(GmmParams g, RowSrc src,
                                                 float* __restrict__ eps) {
    const int groups = src.active ? *src.active : src.max_groups;
    const int64_t rows = (int64_t)groups * src.group;
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    const int gi = (int)(r / src.group), b = (int)(r % src.group);
    const int64_t sl = src.slot ? src.slot[gi] : gi;
    const float* x = src.base + sl * src.slot_stride + (int64_t)b * 2;
    float e0, e1;
    gmm_eps_row(g, row_timestep(src, gi), x[0], x[1], e0, e1);
    eps[r * 2] = e0;
    eps[r * 2 + 1] = e1;
}

__device__ __forceinline__ float drift(float A, float x, float B, float e) {
    return __fadd_rn(__fmul_rn(A, x), __fmul_rn(B, e));
}

// Inclusive prefix sum over the 64 lanes of a wave (every lane active): four
// shift-right steps give the running sum within each row of 16 lanes (lanes
// whose source lies before the row start add zero), then the last lane of
// row 0 is added to row 1 and that of row 2 to row 3, and lane 31 (the total
// of rows 0 and 1) to rows 2 and 3.  The additions are fixed, so the result
// does not depend on timing.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_or_zero(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 ROW_MASK, 0xf, true));
}
__device__ __forceinline__ float wave_prefix_sum(float v) {
    v = __fadd_rn(v, dpp_or_zero<0x111, 0xf>(v));   // row_shr:1
    v = __fadd_rn(v, dpp_or_zero<0x112, 0xf>(v));   // row_shr:2
    v = __fadd_rn(v, dpp_or_zero<0x114, 0xf>(v));   // row_shr:4
    v = __fadd_rn(v, dpp_or_zero<0x118, 0xf>(v));   // row_shr:8
    v = __fadd_rn(v, dpp_or_zero<0x142, 0xa>(v));   // row_bcast:15 into rows 1, 3
    v = __fadd_rn(v, dpp_or_zero<0x143, 0xc>(v));   // row_bcast:31 into rows 2, 3
    return v;
}

// Per trajectory index i, everything one step needs, staged in LDS by every
// thread of the workgroup: drift coefficients, tolerance variance and the
// network-timestep constants of the mixture's eps, plus the component means.
struct GmmStepTables {
    float *A, *B, *V, *a, *inv2s2, *coef, *means;
};

__device__ __forceinline__ float* gmm_stage(const GmmLoopArgs& g, float* sm, GmmStepTables& t) {
    const int T = g.T, K = g.g.K;
    t.A = sm;
    t.B = t.A + T;
    t.V = t.B + T;
    t.a = t.V + T;
    t.inv2s2 = t.a + T;
    t.coef = t.inv2s2 + T;
    t.means = t.coef + T;
    for (int i = threadIdx.x; i < T; i += blockDim.x) {
        const int n = g.model_t[i];
        t.A[i] = g.A[i];
        t.B[i] = g.B[i];
        t.V[i] = g.tol_var ? g.tol_var[i] : 0.f;
        t.a[i] = g.g.a[n];
        t.inv2s2[i] = g.g.inv2s2[n];
        t.coef[i] = g.g.coef[n];
    }
    for (int i = threadIdx.x; i < 2 * K; i += blockDim.x) t.means[i] = g.g.means[i];
    return t.means + 2 * K;
}

// Algorithm 1 for the 2-D mixture in one workgroup, start to finish: the
// step tables, the window ring, the drift batch, the new points and the
// noise live in LDS, the loop state in registers, and one launch runs every
// iteration.  Drifts are formed in parallel; each column's running sums are
// then taken by one wave as a prefix sum when no wave has more than two
// columns, else by one thread in order along the window.  With `noise_in_lds`
// all T noise vectors are staged once, else each window's are read from HBM.
template <class M>
__global__ __launch_bounds__(1024) void k_gmm_picard_loop(GmmLoopArgs a, int noise_in_lds, GmmDraw draw) {
    extern __shared__ float sm[];
    const int B = a.batch, P1 = a.p + 1, BD = 2 * B, T = a.T;
    GmmStepTables tb;
    float* ring = gmm_stage(a, sm, tb);         // [p+1][B][2]
    float* y = ring + P1 * BD;                  // [p][B][2] drifts
    float* xn = y + a.p * BD;                   // [p][B][2] new points x^{k+1}_{t+j+1}
    float* zw = xn + a.p * BD;                  // noise: [T][B][2] or a [p][B][2] window
    __shared__ int s_stride, s_bad;
    const int tid = threadIdx.x, nth = blockDim.x;
    const int K = a.g.K;
    // the window's running sums: a wave per column when every wave has at
    // most two columns (the block is whole waves), else a thread per column
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), nwaves = nth / 64;
    const bool wave_scan = BD <= 2 * nwaves;
    // the components of a row over four lanes when the block has four
    // threads for every row of a full window (gmm_loop_threads)
    const bool quad = 4 * a.p * B <= nth;
    M mu;
    if constexpr (M::kBound > 0) mu.load(a.g.means, K);
    else mu.p = tb.means;
    if (draw.on) {
        // x_0 (stream 0) into ring slot 0 and every step's noise (stream 1)
        // into LDS, four values per counter block
        const int nq0 = (BD + 3) / 4, nq1 = (T * BD + 3) / 4;
        for (int q = tid; q < nq0 + (draw.zstd ? nq1 : 0); q += nth) {
            const bool prior = q < nq0;
            const int qq = prior ? q : q - nq0;
            float v[4];
            normals4(draw.seed, prior ? 0u : 1u, qq, v);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = 4 * qq + e;
                if (prior && i < BD) ring[i] = v[e];
                if (!prior && i < T * BD) zw[i] = draw.zstd[i / BD] * v[e];
            }
        }
        if (!draw.zstd)
            for (int i = tid; i < T * BD; i += nth) zw[i] = 0.f;
    } else {
        for (int i = tid; i < BD; i += nth) ring[i] = a.x0[i];
        if (noise_in_lds)
            for (int i = tid; i < T * BD; i += nth) zw[i] = a.noise ? a.noise[i] : 0.f;
    }
    int t = 0, k = 0, f = 0;
    int pe = a.p < T ? a.p : T;
    int64_t evals = 0;
    int first_stride = 0;
    if (tid == 0) s_bad = 0;
    __syncthreads();
    while (t < T) {
        // drift batch (network evaluations) and, if not staged, the noise window
        if (!noise_in_lds)
            for (int i = tid; i < pe * BD; i += nth)
                zw[i] = a.noise ? a.noise[(int64_t)t * BD + i] : 0.f;
        if (quad) {
            // four lanes per window row (the launcher gives four threads a row)
            for (int r = tid >> 2; r < pe * B; r += nth >> 2) {
                const int j = r / B, b = r % B, m = t + j;
                const float* x = ring + ((m <= f ? m : f) % P1) * BD + 2 * b;
                float e0, e1;
                gmm_eps_quad(tb.means, K, tid & 3, tb.a[m], tb.inv2s2[m], tb.coef[m], x[0], x[1], e0, e1);
                if ((tid & 3) == 0) {
                    y[r * 2] = drift(tb.A[m], x[0], tb.B[m], e0);
                    y[r * 2 + 1] = drift(tb.A[m], x[1], tb.B[m], e1);
                }
            }
        } else {
            for (int r = tid; r < pe * B; r += nth) {
                const int j = r / B, b = r % B, m = t + j;
                const float* x = ring + ((m <= f ? m : f) % P1) * BD + 2 * b;
                float e0, e1;
                gmm_eps_core(mu, K, tb.a[m], tb.inv2s2[m], tb.coef[m], x[0], x[1], e0, e1);
                y[r * 2] = drift(tb.A[m], x[0], tb.B[m], e0);
                y[r * 2 + 1] = drift(tb.A[m], x[1], tb.B[m], e1);
            }
        }
        if (tid == 0) s_stride = pe;
        __syncthreads();
        // Picard update: x_t + running sum of drifts + running sum of noise
        const float* z = noise_in_lds ? zw + t * BD : zw;
        if (wave_scan) {
            // one wave per column: the running sums of 64 rows at a time as a
            // wave prefix sum, carried from one run of rows to the next
            for (int c = wave; c < BD; c += nwaves) {
                const float anchor = ring[(t % P1) * BD + c];
                float cy = 0.f, cz = 0.f;
                for (int j0 = 0; j0 < pe; j0 += 64) {
                    const int j = j0 + lane;
                    const bool in = j < pe;
                    const float sy = __fadd_rn(cy, wave_prefix_sum(in ? y[j * BD + c] : 0.f));
                    const float sz = __fadd_rn(cz, wave_prefix_sum(in ? z[j * BD + c] : 0.f));
                    if (in) xn[j * BD + c] = __fadd_rn(__fadd_rn(anchor, sy), sz);
                    cy = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sy), 63));
                    cz = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sz), 63));
                }
            }
        } else {
            // one thread per column, in order along the window
            for (int c = tid; c < BD; c += nth) {
                const float anchor = ring[(t % P1) * BD + c];
                float sy = 0.f, sz = 0.f;
#pragma unroll 8
                for (int j = 0; j < pe; ++j) {
                    sy = __fadd_rn(sy, y[j * BD + c]);
                    sz = __fadd_rn(sz, z[j * BD + c]);
                    xn[j * BD + c] = __fadd_rn(__fadd_rn(anchor, sy), sz);
                }
            }
        }
        __syncthreads();
        // errors of offsets o in [1, pe), one thread per (o, b)
        for (int r = tid; r < (pe - 1) * B; r += nth) {
            const int o = 1 + r / B, b = r % B, m = t + o;
            const float* xo = ring + ((m <= f ? m : f) % P1) * BD + 2 * b;
            const float* xv = xn + (o - 1) * BD + 2 * b;
            const float d0 = __fsub_rn(xv[0], xo[0]), d1 = __fsub_rn(xv[1], xo[1]);
            const float err = __fadd_rn(d0 * d0, d1 * d1) / a.err_div;
            const float s2 = tb.V[m + a.tol_offset];
            const float tol = (s2 == 0.f) ? 0.f : a.tau2 * s2;
            if (!isfinite(err)) atomicOr(&s_bad, 1);
            // o does not decrease along the lanes of a wave: the lowest
            // failing lane holds the wave's smallest failing offset
            const uint64_t fails = __ballot(!(err <= tol));
            if (fails && __lane_id() == (unsigned)(__ffsll((unsigned long long)fails) - 1))
                atomicMin(&s_stride, o);
        }
        // the last new point is never tested: check it for non-finite values
        for (int c = tid; c < BD; c += nth)
            if (!isfinite(xn[(pe - 1) * BD + c])) atomicOr(&s_bad, 1);
        __syncthreads();
        // slide: the new points enter the ring, the window moves on
        for (int i = tid; i < pe * BD; i += nth) {
            const int j = i / BD, c = i % BD;
            ring[((t + j + 1) % P1) * BD + c] = xn[i];
        }
        const int stride = s_stride;
        const bool bad = s_bad != 0;
        if (tid == 0) a.trace[k] = stride;
        if (k == 0) first_stride = stride;
        evals += pe;
        f = t + pe;
        t += stride;
        ++k;
        pe = a.p < T - t ? a.p : T - t;
        __syncthreads();
        if (bad) break;
    }
    for (int i = tid; i < BD; i += nth) a.out[i] = ring[(T % P1) * BD + i];
    if (tid == 0) {
        LoopState v;
        v.t = t;
        v.k = k;
        v.f = f;
        v.p_eff = 0;
        v.first_stride = first_stride;
        v.nrows = 0;
        v.evals = evals;
        v.status = s_bad ? PD_ERR_NUMERIC : PD_OK;
        *a.st = v;
        mirror_state(v, a.st_host);
    }
}

// The sequential chain for the 2-D mixture in one workgroup, one thread, or
// one quad of four lanes, per sample (its two coordinates never interact with
// other samples).  The noise
// of `chunk` steps at a time is staged in LDS by all threads together.
template <class M>
__global__ __launch_bounds__(1024) void k_gmm_sequential_loop(GmmLoopArgs a, int chunk) {
    extern __shared__ float sm[];
    const int B = a.batch, T = a.T, K = a.g.K;
    const int tid = threadIdx.x, nth = blockDim.x;
    GmmStepTables tb;
    float* zs = gmm_stage(a, sm, tb);  // [chunk][samples of this pass][2]
    M mu;
    if constexpr (M::kBound > 0) mu.load(a.g.means, K);
    else mu.p = tb.means;
    // the components of a sample over four lanes when the block has four
    // threads for every sample (gmm_loop_threads)
    const bool quad = 4 * B <= nth;
    const int per = quad ? nth >> 2 : nth, me = quad ? tid >> 2 : tid;   // samples per pass
    for (int b0 = 0; b0 < B; b0 += per) {
        const int nb = B - b0 < per ? B - b0 : per, b = b0 + me;
        const bool active = me < nb;
        float x0 = 0.f, x1 = 0.f;
        if (active) {
            x0 = a.x0[2 * b];
            x1 = a.x0[2 * b + 1];
        }
        for (int i0 = 0; i0 < T; i0 += chunk) {
            const int n = T - i0 < chunk ? T - i0 : chunk;
            __syncthreads();
            for (int q = tid; q < n * 2 * nb; q += nth) {
                const int ii = q / (2 * nb), r = q % (2 * nb);
                zs[q] = a.noise ? a.noise[((int64_t)(i0 + ii) * B + b0) * 2 + r] : 0.f;
            }
            __syncthreads();
            if (!active) continue;
            for (int ii = 0; ii < n; ++ii) {
                const int i = i0 + ii;
                float e0, e1;
                if (quad)
                    gmm_eps_quad(tb.means, K, tid & 3, tb.a[i], tb.inv2s2[i], tb.coef[i], x0, x1, e0, e1);
                else
                    gmm_eps_core(mu, K, tb.a[i], tb.inv2s2[i], tb.coef[i], x0, x1, e0, e1);
                const float* z = zs + (ii * nb + me) * 2;
                const float v0 = __fadd_rn(__fadd_rn(x0, drift(tb.A[i], x0, tb.B[i], e0)), z[0]);
                const float v1 = __fadd_rn(__fadd_rn(x1, drift(tb.A[i], x1, tb.B[i], e1)), z[1]);
                x0 = v0;
                x1 = v1;
            }
        }
        if (active && (!quad || (tid & 3) == 0)) {
            a.out[2 * b] = x0;
            a.out[2 * b + 1] = x1;
        }
    }
}

// Threads of the two loops: four per row of a full window (Picard) or per
// sample (sequential) when that fits one workgroup, else one.
static int gmm_loop_threads(int64_t rows) {
    const int64_t t = 4 * rows <= 1024 ? 4 * rows : rows;
    return t < 1024 ? (int)((t + 63) / 64) * 64 : 1024;
}

}  // namespace

// LDS of the fused Picard loop: step tables, ring, drifts, new points and a
// noise window; the whole noise takes (T - p) more windows' worth.
static size_t picard_loop_floats(int T, int K, int p, int batch, bool noise_in_lds) {
    const size_t BD = 2 * (size_t)batch;
    return 6 * (size_t)T + 2 * (size_t)K + BD * ((size_t)(p + 1) + 2 * (size_t)p) +
           BD * (noise_in_lds ? (size_t)T : (size_t)p);
}

size_t gmm_loop_lds_bytes(int T, int K, int p, int batch) {
    return sizeof(float) * picard_loop_floats(T, K, p, batch, false);
}

bool gmm_loop_stages_noise(int T, int K, int p, int batch, size_t max_lds) {
    return sizeof(float) * picard_loop_floats(T, K, p, batch, true) <= max_lds;
}

void launch_gmm_picard_loop(const GmmLoopArgs& a, size_t max_lds, hipStream_t s) {
    launch_gmm_picard_loop(a, GmmDraw{0, 0, nullptr}, max_lds, s);
}

void launch_gmm_picard_loop(const GmmLoopArgs& a, const GmmDraw& draw, size_t max_lds,
                            hipStream_t s) {
    if (a.g.K > kMaxK) fail(PD_ERR_UNSUPPORTED, "gmm2d supports at most 64 components");
    const size_t full = sizeof(float) * picard_loop_floats(a.T, a.g.K, a.p, a.batch, true);
    const bool noise_in_lds = full <= max_lds;
    if (draw.on && !noise_in_lds)
        fail(PD_ERR_INVALID_ARG, "gmm2d loop: drawing the noise in the loop needs it all in LDS");
    const size_t lds = noise_in_lds ? full : gmm_loop_lds_bytes(a.T, a.g.K, a.p, a.batch);
    // enough waves for one drift per four threads (or per thread): fewer
    // waves meet at the barriers
    const int threads = gmm_loop_threads((int64_t)a.p * a.batch);
    if (a.g.K <= 8)
        hipLaunchKernelGGL(k_gmm_picard_loop<MeansReg<8>>, dim3(1), dim3(threads), lds, s, a,
                           (int)noise_in_lds, draw);
    else if (a.g.K <= 16)
        hipLaunchKernelGGL(k_gmm_picard_loop<MeansReg<16>>, dim3(1), dim3(threads), lds, s, a,
                           (int)noise_in_lds, draw);
    else
        hipLaunchKernelGGL(k_gmm_picard_loop<MeansMem>, dim3(1), dim3(threads), lds, s, a,
                           (int)noise_in_lds, draw);
    PD_HIP(hipGetLastError());
}

void launch_gmm_sequential_loop(const GmmLoopArgs& a, hipStream_t s) {
    if (a.g.K > kMaxK) fail(PD_ERR_UNSUPPORTED, "gmm2d supports at most 64 components");
    const int threads = gmm_loop_threads(a.batch);
    const int per_step = 2 * (a.batch < threads ? a.batch : threads);
    const size_t tables = sizeof(float) * (6 * (size_t)a.T + 2 * (size_t)a.g.K);
    if (tables + sizeof(float) * per_step > kLoopLdsMax)
        fail(PD_ERR_UNSUPPORTED, "schedule too long for the single-workgroup loop");
    size_t chunk = (kLoopLdsMax - tables) / (sizeof(float) * per_step);
    chunk = chunk > (size_t)a.T ? (size_t)a.T : chunk;
    const size_t lds = tables + sizeof(float) * chunk * per_step;
    if (a.g.K <= 8)
        hipLaunchKernelGGL(k_gmm_sequential_loop<MeansReg<8>>, dim3(1), dim3(threads), lds, s, a,
                           (int)chunk);
    else if (a.g.K <= 16)
        hipLaunchKernelGGL(k_gmm_sequential_loop<MeansReg<16>>, dim3(1), dim3(threads), lds, s, a,
                           (int)chunk);
    else
        hipLaunchKernelGGL(k_gmm_sequential_loop<MeansMem>, dim3(1), dim3(threads), lds, s, a,
                           (int)chunk);
    PD_HIP(hipGetLastError());
}

void launch_gmm_eps(const GmmParams& g, const RowSrc& src, float* eps, hipStream_t s) {
    if (g.K > kMaxK) fail(PD_ERR_UNSUPPORTED, "gmm2d supports at most 64 components");
    const int64_t rows = (int64_t)src.max_groups * src.group;
    if (rows == 0) return;
    hipLaunchKernelGGL(k_gmm_eps, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, g, src,
                       eps);
    PD_HIP(hipGetLastError());
}

}  // namespace pd
