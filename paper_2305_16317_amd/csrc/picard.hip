// Picard update, error check and window slide of Algorithm 1 on the device.
//
// The window x_t .. x_{t+p} lives in a ring of p+1 trajectory slots,
// slot(m) = m mod (p+1).  The frontier f is the highest index that holds a
// computed point; every point past f equals x_f (the new points of Algorithm
// 1 are copies of the window's last point), so they are read from slot(f)
// and never copied.  The loop state (t, k, f, p_eff) stays on the device: the
// finalize kernel of one iteration writes the row descriptors (ring slot and
// network timestep of every window point) that the next iteration's denoiser
// and scan read, so no host round trip is needed between iterations.
#include "pd_internal.h"

namespace pd {
namespace {

constexpr int kScanWaves = 4;             // waves per scan block, split along the window
constexpr int kScanCols = 64;             // columns (sample elements) per scan block
constexpr int kScanMaxRows = 32;          // rows per wave: windows up to 4 * 32 = 128 points
constexpr int kMaxWindow = kScanWaves * kScanMaxRows;

__device__ __forceinline__ float drift(float A, float x, float B, float e) {
    // y = A x + B eps, two products and one sum, each rounded (no contraction)
    return __fadd_rn(__fmul_rn(A, x), __fmul_rn(B, e));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__global__ void k_picard_init(LoopState* st, int32_t* slot, int32_t* nrow,
                              const int32_t* __restrict__ model_t, int T, int p) {
    const int pe = p < T ? p : T;
    if (threadIdx.x == 0) {
        st->t = 0;
        st->k = 0;
        st->f = 0;
        st->p_eff = pe;
        st->status = PD_OK;
        st->first_stride = 0;
        st->evals = 0;
    }
    for (int j = threadIdx.x; j < pe; j += blockDim.x) {
        slot[j] = 0;            // every initial window point is a copy of x_0
        nrow[j] = model_t[j];
    }
}

// Sum each of the R values v[0..R) of a lane over the 64 lanes of the wave.
// Butterfly with halving: at every step a lane keeps half of its values and
// adds the partner's copy of that half, so R - 1 + log2(64/R) shuffles cover
// all R sums (instead of 6 R).  Returns the full sum of value index `idx`
// (a function of the lane); lanes with (lane & (64/R - 1)) == 0 hold distinct
// indices.  Every sum is formed in a fixed order, so results are reproducible.
template <int R>
__device__ __forceinline__ float multi_wave_sum(float (&v)[R], int lane, int& idx) {
    idx = 0;
#pragma unroll
    for (int h = R / 2, bit = 32; h >= 1; h /= 2, bit /= 2) {
        const bool upper = (lane & bit) != 0;
#pragma unroll
        for (int i = 0; i < h; ++i) {
            const float keep = upper ? v[i + h] : v[i];
            const float send = upper ? v[i] : v[i + h];
            v[i] = keep + __shfl_xor(send, bit, 64);
        }
        if (upper) idx += h;
    }
    float r = v[0];
#pragma unroll
    for (int bit = 32 / R; bit >= 1; bit /= 2) r += __shfl_xor(r, bit, 64);
    return r;
}

// One block: 64 columns of one sample b, all window rows, split over 4 waves
// (rows [w*ch, (w+1)*ch) per wave, ch <= R).  Drift and noise are summed along
// the rows inside each wave, the wave totals are exchanged through LDS, and
// the new points x^{k+1}_{t+j+1} = x_t + sum y + sum z are written back to the
// ring.  All loads use clamped, always-valid indices and no branches, so the
// R rows' loads of a wave are in flight together.  The squared differences
// against the old points are reduced over the 64 columns per window offset
// and written as per-block partial sums partials[b][o][blk]; offset 0 (never
// tested) carries the count of non-finite new points instead.
template <int R, bool NOISE>
__global__ __launch_bounds__(256) void k_picard_scan(
    const LoopState* __restrict__ st, float* ring, const float* __restrict__ eps,
    const float* __restrict__ noise, const float* __restrict__ Atab,
    const float* __restrict__ Btab, int p, int batch, int64_t D, float* __restrict__ partials) {
    const int pe = st->p_eff;
    if (pe <= 0) return;
    const int t = st->t, f = st->f;
    // the wave index is uniform: keep it (and every row index derived from
    // it) in scalar registers so the per-row table reads are scalar loads
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int b = blockIdx.y, blk = blockIdx.x, nblk = gridDim.x;
    const int64_t d = (int64_t)blk * kScanCols + lane;
    const bool valid = d < D;
    const int64_t slotsz = (int64_t)batch * D;
    const int64_t col = (int64_t)b * D + (valid ? d : 0);
    const int P1 = p + 1;
    const int ch = (pe + kScanWaves - 1) / kScanWaves;
    const int j0 = min(w * ch, pe), j1 = min(j0 + ch, pe);
    const int nr = j1 - j0;

    __shared__ float s_tot[2][kScanWaves][kScanCols];
    __shared__ float s_first[kScanWaves][kScanCols];
    __shared__ float s_bad[kScanWaves];

    // ---- every read of this block's ring columns is consumed before the
    // barrier; the writes all come after it (the ring slots overlap).
    const float anchor = ring[(int64_t)(t % P1) * slotsz + col];
    const int slot_f = f % P1;
    float xo[R], e[R], z[R], ca[R], cb[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = min(j0 + r, pe - 1);            // clamped: always a window row
        const int m = t + j;
        const int sl = m <= f ? m % P1 : slot_f;      // points past f equal x_f
        xo[r] = ring[(int64_t)sl * slotsz + col];
        e[r] = eps[(int64_t)j * slotsz + col];
        z[r] = NOISE ? noise[(int64_t)m * slotsz + col] : 0.f;
        ca[r] = Atab[m];
        cb[r] = Btab[m];
    }
    // drifts of every (clamped) row first, then the masked running sums: no
    // load is left behind a condition
    float y[R];
#pragma unroll
    for (int r = 0; r < R; ++r) y[r] = drift(ca[r], xo[r], cb[r], e[r]);
    float sy[R], sz[R];
    float acc_y = 0.f, acc_z = 0.f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool in = r < nr;
        acc_y = __fadd_rn(acc_y, in ? y[r] : 0.f);
        acc_z = __fadd_rn(acc_z, in ? z[r] : 0.f);
        sy[r] = acc_y;
        sz[r] = acc_z;
    }
    s_tot[0][w][lane] = acc_y;
    s_tot[1][w][lane] = acc_z;
    s_first[w][lane] = xo[0];       // x^k_{t+j0}: the next wave's old point past its range
    __syncthreads();
    float py = 0.f, pz = 0.f;
    for (int v = 0; v < w; ++v) {
        py = __fadd_rn(py, s_tot[0][v][lane]);
        pz = __fadd_rn(pz, s_tot[1][v][lane]);
    }
    const float next_old = (w + 1 < kScanWaves) ? s_first[w + 1][lane] : 0.f;

    // ---- new points, their errors, and the writes
    float bad = 0.f, d2[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = j0 + r;
        const float xn = __fadd_rn(__fadd_rn(anchor, __fadd_rn(py, sy[r])), __fadd_rn(pz, sz[r]));
        const bool in = r < nr;
        if (in && valid) {
            ring[(int64_t)((t + j + 1) % P1) * slotsz + col] = xn;
            bad += isfinite(xn) ? 0.f : 1.f;
        }
        // error of window offset o = j + 1: x^{k+1}_{t+j+1} against x^k_{t+j+1}
        const float xold = (r + 1 < R && r + 1 < nr) ? xo[r + 1 < R ? r + 1 : r] : next_old;
        const float dl = (in && valid && j + 1 < pe) ? __fsub_rn(xn, xold) : 0.f;
        d2[r] = dl * dl;
    }
    int idx;
    const float s = multi_wave_sum<R>(d2, lane, idx);
    if ((lane & (64 / R - 1)) == 0 && idx < nr && j0 + idx + 1 < pe)
        partials[((int64_t)b * p + j0 + idx + 1) * nblk + blk] = s;
    bad = wave_sum(bad);
    if (lane == 0) s_bad[w] = bad;
    __syncthreads();
    if (threadIdx.x == 0) {
        float nb = 0.f;
        for (int v = 0; v < kScanWaves; ++v) nb += s_bad[v];
        partials[((int64_t)b * p + 0) * nblk + blk] = nb;
    }
}

// One block: reduce the partials of every (offset, sample), apply the stride
// rule, slide the window and prepare the next iteration's row descriptors.
__global__ __launch_bounds__(1024) void k_picard_finalize(
    LoopState* st, const float* __restrict__ partials, int nblk, int p, int batch, int64_t D,
    int T, const float* __restrict__ tol_var, float tau2, int tol_offset,
    const int32_t* __restrict__ model_t, int32_t* trace, int32_t* slot, int32_t* nrow) {
    const int pe = st->p_eff;
    if (pe <= 0) return;
    const int t = st->t, k = st->k;
    __shared__ int s_stride, s_bad;
    if (threadIdx.x == 0) {
        s_stride = pe;
        s_bad = 0;
    }
    __syncthreads();
    constexpr int kTeam = 16;
    const int team = threadIdx.x / kTeam, tl = threadIdx.x % kTeam;
    const int nteams = blockDim.x / kTeam;
    const float Df = (float)D;
    for (int pair = team; pair < pe * batch; pair += nteams) {
        const int o = pair / batch, b = pair % batch;
        const float* src = partials + ((int64_t)b * p + o) * nblk;
        // 8 independent loads per step keep the team's reads in flight together
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (int i0 = 0; i0 < nblk; i0 += 8 * kTeam) {
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int i = i0 + u * kTeam + tl;
                acc[u] += i < nblk ? src[i] : 0.f;
            }
        }
        float s = ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
#pragma unroll
        for (int off = kTeam / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, kTeam);
        if (tl == 0) {
            if (o == 0) {
                if (s != 0.f) atomicOr(&s_bad, 1);
            } else {
                const float err = s / Df;
                if (!isfinite(err)) atomicOr(&s_bad, 1);
                const float s2 = tol_var[t + o + tol_offset];
                const float tol = (s2 == 0.f) ? 0.f : tau2 * s2;
                if (!(err <= tol)) atomicMin(&s_stride, o);
            }
        }
    }
    __syncthreads();
    const int stride = s_stride;
    const int fn = t + pe, tn = t + stride;
    const int pn = s_bad ? 0 : (p < T - tn ? p : T - tn);
    if (threadIdx.x == 0) {
        trace[k] = stride;
        if (k == 0) st->first_stride = stride;
        st->k = k + 1;
        st->evals += pe;
        st->f = fn;
        st->t = s_bad ? T : tn;
        st->p_eff = pn > 0 ? pn : 0;
        if (s_bad) st->status = PD_ERR_NUMERIC;
    }
    for (int j = threadIdx.x; j < pn; j += blockDim.x) {
        const int m = tn + j;
        slot[j] = (m < fn ? m : fn) % (p + 1);
        nrow[j] = model_t[m];
    }
}

__global__ __launch_bounds__(256) void k_seq_step(float* __restrict__ x,
                                                  const float* __restrict__ eps,
                                                  const float* __restrict__ z, float A, float B,
                                                  int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float v = __fadd_rn(x[i], drift(A, x[i], B, eps[i]));
    if (z) v = __fadd_rn(v, z[i]);
    x[i] = v;
}

}  // namespace

int picard_partial_blocks(int64_t D) { return (int)((D + kScanCols - 1) / kScanCols); }

void launch_picard_init(LoopState* st, int32_t* slot, int32_t* nrow, const int32_t* model_t,
                        int T, int p, hipStream_t s) {
    hipLaunchKernelGGL(k_picard_init, dim3(1), dim3(256), 0, s, st, slot, nrow, model_t, T, p);
    PD_HIP(hipGetLastError());
}

void launch_picard_scan(const LoopState* st, float* ring, const float* eps, const float* noise,
                        const float* A, const float* B, int p, int batch, int64_t D,
                        float* partials, hipStream_t s) {
    if (p > kMaxWindow) fail(PD_ERR_UNSUPPORTED, "window larger than 128 points");
    const dim3 grid((unsigned)picard_partial_blocks(D), (unsigned)batch);
    const int ch = (p + kScanWaves - 1) / kScanWaves;    // rows per wave at a full window
#define PD_SCAN(R)                                                                           \
    if (ch <= R) {                                                                           \
        if (noise)                                                                           \
            hipLaunchKernelGGL((k_picard_scan<R, true>), grid, dim3(kScanWaves * 64), 0, s, st, \
                               ring, eps, noise, A, B, p, batch, D, partials);               \
        else                                                                                 \
            hipLaunchKernelGGL((k_picard_scan<R, false>), grid, dim3(kScanWaves * 64), 0, s,    \
                               st, ring, eps, noise, A, B, p, batch, D, partials);           \
        PD_HIP(hipGetLastError());                                                           \
        return;                                                                              \
    }
    PD_SCAN(1) PD_SCAN(2) PD_SCAN(4) PD_SCAN(8) PD_SCAN(16) PD_SCAN(32)
#undef PD_SCAN
    PD_HIP(hipGetLastError());
}

void launch_picard_finalize(LoopState* st, const float* partials, int p, int batch, int64_t D,
                            int T, const float* tol_var, float tau2, int tol_offset,
                            const int32_t* model_t, int32_t* trace, int32_t* slot,
                            int32_t* nrow, hipStream_t s) {
    hipLaunchKernelGGL(k_picard_finalize, dim3(1), dim3(1024), 0, s, st, partials,
                       picard_partial_blocks(D), p, batch, D, T, tol_var, tau2, tol_offset,
                       model_t, trace, slot, nrow);
    PD_HIP(hipGetLastError());
}

void launch_seq_step(float* x, const float* eps, const float* z, float A, float B, int64_t n,
                     hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_seq_step, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x, eps, z,
                       A, B, n);
    PD_HIP(hipGetLastError());
}

}  // namespace pd
