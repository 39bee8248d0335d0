// Picard update, error check and window slide of Algorithm 1 on the device.
//
// The window x_t .. x_{t+p} lives in a ring of p+1 trajectory slots,
// slot(m) = m mod (p+1) (p+2 for the multistep drift, which also keeps
// x_{t-1}).  The frontier f is the highest index that holds a computed
// point; every point past f equals x_f (the new points of Algorithm 1 are
// copies of the window's last point), so they are read from slot(f) and
// never copied.  The loop state (t, k, f, p_eff) stays on the device: the
// finalize step of one iteration writes the row descriptors (ring slot and
// network timestep of every window point) that the next iteration's denoiser
// and scan read, so no host round trip is needed between iterations; it also
// copies the state into mapped host memory for the host's batch decisions.
#include <type_traits>

#include "linear_tile.h"
#include "pd_internal.h"

namespace pd {
namespace {

// Waves per scan block, split along the window: 8 for windows of up to 64
// points, 16 above (up to 8 rows per wave, so windows up to 128 points).  At
// 64 points and 4 x 4 x 96 x 96 columns, 8 waves of 8 rows took 20.8 us per
// launch against 25.3 us for 16 waves of 4; 16 rows per wave spill.
constexpr int kScanMaxRows = 8;
constexpr int kMaxWindow = 16 * kScanMaxRows;

// Columns per lane of the scan: four (one 16-byte access per row) when the
// sample size allows it, else one.
inline int scan_vec(int64_t D) { return D % 4 == 0 ? 4 : 1; }

template <int VEC>
struct Cols;
template <>
struct Cols<1> {
    typedef float type;
};
template <>
struct Cols<4> {
    typedef float type __attribute__((ext_vector_type(4)));
};
template <int VEC>
__device__ __forceinline__ float& col_at(typename Cols<VEC>::type& v, int c) {
    if constexpr (VEC == 1) return v;
    else return reinterpret_cast<float*>(&v)[c];
}
template <int VEC>
__device__ __forceinline__ float col_at(const typename Cols<VEC>::type& v, int c) {
    if constexpr (VEC == 1) return v;
    else return v[c];
}

// Sum over aligned groups of N lanes (N a power of two <= 64); every lane of
// a group ends with the group's sum.  Groups up to 16 lanes reduce with DPP
// lane moves inside a row (quad swaps, then the 8- and 16-lane mirrors), with
// no LDS traffic; wider groups finish with a cross-row shuffle.
template <int N>
__device__ __forceinline__ float group_sum(float v) {
    auto dpp = [](float x, auto ctrl) {
        return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                             0, __builtin_bit_cast(int, x), decltype(ctrl)::value,
                                             0xF, 0xF, false));
    };
    if constexpr (N >= 2) v += dpp(v, std::integral_constant<int, 0xB1>{});   // quad_perm [1,0,3,2]
    if constexpr (N >= 4) v += dpp(v, std::integral_constant<int, 0x4E>{});   // quad_perm [2,3,0,1]
    if constexpr (N >= 8) v += dpp(v, std::integral_constant<int, 0x141>{});  // row_half_mirror
    if constexpr (N >= 16) v += dpp(v, std::integral_constant<int, 0x140>{}); // row_mirror
    if constexpr (N >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (N >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

__device__ __forceinline__ float drift(float A, float x, float B, float e) {
    // y = A x + B eps, two products and one sum, each rounded (no contraction)
    return __fadd_rn(__fmul_rn(A, x), __fmul_rn(B, e));
}

// Heun's method, window side (rows j < p_eff of the current window):
// predict:  xt[j] = x_{t+j} + (A x_{t+j} + B eps[j])      (the Euler step)
// The scan then takes (eps[j] + eps2[j]) / 2 in place of eps[j] for every step
// but the last, so that its A x + B eps is A x + (B / 2)(eps + eps2) rounded
// exactly as written (halving is exact).
__global__ __launch_bounds__(256) void k_heun_predict(const LoopState* __restrict__ st,
                                                      const float* __restrict__ ring,
                                                      const float* __restrict__ eps,
                                                      const float* __restrict__ Atab,
                                                      const float* __restrict__ Btab, int p,
                                                      int64_t BD, float* __restrict__ xt) {
    const int pe = st->p_eff;
    const int t = st->t, f = st->f, P1 = p + 1;
    const int64_t n = (int64_t)pe * BD;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int j = (int)(i / BD);
        const int64_t c = i - (int64_t)j * BD;
        const int m = t + j;
        const float x = ring[(int64_t)((m <= f ? m : f) % P1) * BD + c];
        xt[i] = __fadd_rn(x, drift(Atab[m], x, Btab[m], eps[i]));
    }
}


// Barrier for LDS traffic only: global stores issued before it need not have
// completed (later kernels read them, no wave of this block does).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The stride is known: record it, slide the window and write the next
// iteration's row descriptors.  cur is the loop state as the iteration found
// it.  mt / mt2 (or nullptr: read the tables) hold model_t[t + i] /
// model_t_next[t + i] for i < 2p, which covers every index read here (the
// next window starts at t + stride <= t + p_eff).  Thread 0 rewrites the loop
// state.
__device__ void finalize_apply(const FinalizeArgs& a, int stride, int bad, const LoopState& cur,
                               const int* mt, const int* mt2) {
    LoopState* st = a.st;
    const int p = a.p, T = a.T;
    const int t = cur.t, k = cur.k, pe = cur.p_eff, rows_now = cur.nrows;
    const int fn = t + pe, tn = t + stride;
    const int pn = bad ? 0 : (p < T - tn ? p : T - tn);
    auto model_t = [&](int m) { return mt ? mt[m - t] : a.model_t[m]; };
    auto model_t_next = [&](int m) { return mt2 ? mt2[m - t] : a.model_t_next[m]; };
    // next batch: [the point before the window, for the multistep drift] then
    // the window's points
    const int hn = (a.history && tn >= 1 && pn > 0) ? 1 : 0;
    if (threadIdx.x == 0) {
        a.trace[k] = stride;
        LoopState v = cur;
        if (k == 0) v.first_stride = stride;
        v.k = k + 1;
        // network evaluations: Heun evaluates twice per point but the last
        // step; with a history row the batch had one row more than the window
        v.evals += a.nrow2 ? 2 * pe - (t + pe == T ? 1 : 0) : rows_now;
        v.f = fn;
        v.t = bad ? T : tn;
        v.p_eff = pn > 0 ? pn : 0;
        if (bad) v.status = PD_ERR_NUMERIC;
        v.nrows = pn > 0 ? pn + hn : 0;
        *st = v;
        if (hn) {
            a.slot[0] = (tn - 1) % a.ring_slots;     // tn - 1 < fn: a computed point
            a.nrow[0] = model_t(tn - 1);
        }
        mirror_state(v, a.st_host);
    }
    for (int j = threadIdx.x; j < pn; j += blockDim.x) {
        const int m = tn + j;
        a.slot[hn + j] = (m < fn ? m : fn) % a.ring_slots;
        a.nrow[hn + j] = model_t(m);
        if (a.nrow2) a.nrow2[j] = model_t_next(m);
    }
    // the iteration that reaches T copies x_T out, so the host needs no copy
    // launch: its new points are this block's own stores (waited for here) or
    // were made visible to it by kernel order or the count-in.  The condition
    // is uniform over the block.
    if (!bad && tn >= T) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        for (int64_t i = threadIdx.x; i < a.BD; i += blockDim.x) a.x_out[i] = a.xT[i];
    }
}

// Tolerance of window offset o >= 1 (Algorithm 1's stride test compares the
// error with it; sigma^2 = 0 allows no change at all).
__device__ __forceinline__ float offset_tol(const FinalizeArgs& a, int t, int o) {
    const float s2 = a.tol_var[t + o + a.tol_offset];
    return (s2 == 0.f) ? 0.f : a.tau2 * s2;
}

// One block: reduce the partials of every (offset, sample), apply the stride
// rule, slide the window and prepare the next iteration's row descriptors.
// cur is the loop state as the iteration found it; thread 0 rewrites it at
// the end.
__device__ void finalize_body(const FinalizeArgs& a, int nblk, const LoopState& cur) {
    const int pe = cur.p_eff;
    if (pe <= 0) return;
    const int t = cur.t, p = a.p;
    __shared__ int s_stride, s_bad;
    if (threadIdx.x == 0) {
        s_stride = pe;
        s_bad = 0;
    }
    __syncthreads();
    constexpr int kTeam = 16;
    const int team = threadIdx.x / kTeam, tl = threadIdx.x % kTeam;
    const int nteams = blockDim.x / kTeam;
    for (int pair = team; pair < pe * a.batch; pair += nteams) {
        const int o = pair / a.batch, b = pair % a.batch;
        const float tol = o >= 1 ? offset_tol(a, t, o) : 0.f;    // in flight with the sums
        const float* src = a.partials + ((int64_t)b * p + o) * nblk;
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
        s = group_sum<kTeam>(s);
        bool fails = false, bad = false;
        if (tl == 0) {
            if (o == 0) {
                bad = s != 0.f;
            } else {
                const float err = s / a.err_div;
                bad = !isfinite(err);
                fails = !(err <= tol);
            }
        }
        // lanes hold pairs in increasing order: the wave's first failing
        // lane has its smallest failing offset, and one lane per wave votes
        const uint64_t fm = __ballot(fails), bm = __ballot(bad);
        const int lane = threadIdx.x & 63;
        if (fm && lane == __ffsll((unsigned long long)fm) - 1) atomicMin(&s_stride, o);
        if (bm && lane == __ffsll((unsigned long long)bm) - 1) atomicOr(&s_bad, 1);
    }
    __syncthreads();
    finalize_apply(a, s_stride, s_bad, cur, nullptr, nullptr);
}

// The finalize step of a multi-block scan (kernel order makes every block's
// partials visible to it).
__global__ __launch_bounds__(1024) void k_picard_finalize(FinalizeArgs a, int nblk) {
    const LoopState cur = *a.st;
    finalize_body(a, nblk, cur);
}

// The MLP's last layer with the Picard update as its epilogue (Euler drift,
// windows of up to kHeadGroups * kHeadRows points).  Each block computes one
// 16 x 16 tile of epsilon exactly as the layer kernel does (linear_tile), then
// counts itself in on its 16-column slab; the slab's last block, which then
// sees every window row of those columns, rebuilds them: drift, running sums
// of drift and noise, new points, and the per-offset squared differences
// summed over its 16 columns into partials[b][o][slab] (offset 0 carries the
// count of non-finite points in the window's last row, as in the scan
// kernel).  The last slab to finish applies the stride rule and slides the
// window (finalize_body).  Nothing waits: a block that is not last returns,
// and a counter is reset by the block that completes it (count_in).  p_eff
// never grows from one iteration to the next, so a block that
// starts after the slide still finds itself past the window and returns.
constexpr int kHeadGroups = kLinWaves * 4;   // 16-lane row groups of the block

// Counts the block in on *cnt, which completes at n arrivals.  Each wave waits
// for its own global stores to reach L2; after the barrier one thread makes the
// block's stores visible device-wide (one L2 write-back per block, not per
// wave) and counts.  The block that completes the count resets it, invalidates
// its caches (so it reads what every counted block stored) and returns true;
// every other block returns false.
__device__ bool count_in(int32_t* cnt, int n) {
    __shared__ int s_flag;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        const int last = atomicAdd(cnt, 1) == n - 1;
        if (last) {
            atomicExch(cnt, 0);                  // where the next launch's arrivals count
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        }
        s_flag = last;
    }
    __syncthreads();
    return s_flag != 0;
}
constexpr int kHeadRows = 4;                 // window rows per group
static_assert(kHeadGroups * kHeadRows >= kMaxWindow, "the head covers every window size");

template <bool NOISE>
__global__ __launch_bounds__(kLinWaves * 64) void k_mlp_head_scan(HeadScanArgs a, FinalizeArgs fin) {
    const LoopState cur = *a.st;
    const int pe = cur.p_eff;
    if (pe <= 0) return;
    const int B = a.batch;
    const int M = pe * B;                        // rows (window point, sample)
    const int slab = blockIdx.x, m0 = blockIdx.y * 16, n0 = slab * 16;
    if (m0 >= M) return;                         // uniform over the block
    linear_tile<false>(a.l4, a.h, a.rows, 0, a.eps, M, m0, n0);

    // the slab's last block rebuilds its columns from every block's epsilon
    if (!count_in(&a.count[slab], (M + 15) / 16)) return;

    const int t = cur.t, f = cur.f, P1 = fin.ring_slots;
    const int64_t D = a.D, BD = (int64_t)B * D;
    const int c = threadIdx.x & 15, g = threadIdx.x >> 4;
    const int ch = (pe + kHeadGroups - 1) / kHeadGroups;          // rows per group
    const int j0 = min(g * ch, pe), nr = min(j0 + ch, pe) - j0;
    const int64_t d = n0 + c;
    const bool valid = d < D;
    const int64_t dc = valid ? d : 0;
    __shared__ float s_tot[2][kHeadGroups][16], s_first[kHeadGroups][16];
    for (int b = 0; b < B; ++b) {
        const int64_t col = (int64_t)b * D + dc;
        // every read of the ring comes before the first barrier; the writes
        // all after it (the ring slots overlap)
        const float anchor = a.ring[(int64_t)(t % P1) * BD + col];
        float xo[kHeadRows], y[kHeadRows], z[kHeadRows];
#pragma unroll
        for (int r = 0; r < kHeadRows; ++r) {
            const int j = min(j0 + r, pe - 1);        // clamped: always a window row
            const int m = t + j;
            const int sl = m <= f ? m % P1 : f % P1;  // points past f equal x_f
            xo[r] = a.ring[(int64_t)sl * BD + col];
            const float e = a.eps[((int64_t)j * B + b) * D + dc];
            y[r] = drift(a.A[m], xo[r], a.B[m], e);
            z[r] = NOISE ? a.noise[(int64_t)m * BD + col] : 0.f;
            if (r >= nr) y[r] = z[r] = 0.f;           // rows past the group's range
        }
        float ty = 0.f, tz = 0.f;
#pragma unroll
        for (int r = 0; r < kHeadRows; ++r) {
            ty = __fadd_rn(ty, y[r]);
            tz = __fadd_rn(tz, z[r]);
        }
        s_tot[0][g][c] = ty;
        s_tot[1][g][c] = tz;
        s_first[g][c] = xo[0];                        // x^k_{t+j0}: the previous group's next old point
        __syncthreads();
        float py = 0.f, pz = 0.f;
        for (int v = 0; v < g; ++v) {
            py = __fadd_rn(py, s_tot[0][v][c]);
            pz = __fadd_rn(pz, s_tot[1][v][c]);
        }
        const float next_old = g + 1 < kHeadGroups ? s_first[g + 1][c] : 0.f;
        float sy = 0.f, sz = 0.f;
#pragma unroll
        for (int r = 0; r < kHeadRows; ++r) {
            const int j = j0 + r;
            const bool in = r < nr;
            sy = __fadd_rn(sy, y[r]);
            sz = __fadd_rn(sz, z[r]);
            const float v = __fadd_rn(__fadd_rn(anchor, __fadd_rn(py, sy)), __fadd_rn(pz, sz));
            // error of window offset o = j + 1: x^{k+1}_{t+j+1} against x^k_{t+j+1}
            const float xold = (r + 1 < kHeadRows && r + 1 < nr) ? xo[r + 1 < kHeadRows ? r + 1 : r] : next_old;
            float e2;
            if (j + 1 < pe) {
                const float dl = __fsub_rn(v, xold);
                e2 = dl * dl;
            } else {
                e2 = isfinite(v) ? 0.f : 1.f;         // last row: count non-finite points
            }
            e2 = (in && valid) ? e2 : 0.f;
            if (in && valid) a.ring[(int64_t)((t + j + 1) % P1) * BD + (int64_t)b * D + d] = v;
            const float s16 = group_sum<16>(e2);      // the slab's 16 columns
            if (in && c == 0)
                a.partials[((int64_t)b * fin.p + (j + 1 < pe ? j + 1 : 0)) * a.n_slabs + slab] = s16;
        }
        __syncthreads();                              // LDS reuse by the next sample
    }

    // the last slab to finish applies the stride rule to every slab's partials
    if (!count_in(&a.count[a.n_slabs], a.n_slabs)) return;
    finalize_body(fin, a.n_slabs, cur);
}


// One block: cpb <= 64 * VEC consecutive columns of one sample b (a multiple
// of VEC, from picard_scan_cols), all window rows,
// split over NW waves (rows [w*ch, (w+1)*ch) per wave, ch <= R).  Drift and
// noise are summed along the rows inside each wave, the wave totals are
// exchanged through LDS, and the new points x^{k+1}_{t+j+1} = x_t + sum y +
// sum z are written back to the ring.  All loads use clamped, always-valid
// indices and no branches, so a wave's rows are in flight together; the drift
// coefficients of a wave's rows come in one vector load and are broadcast
// with readlane.  The squared differences against the old points are summed
// per lane over its columns, transposed through LDS and reduced per window
// offset into per-block partial sums partials[b][o][blk]; offset 0 (never
// tested) carries the count of non-finite points in the window's last row
// (a non-finite point in any other row makes its error non-finite).  With
// DPM, a second-order step's drift also adds R x_{i-1} + S eps_{i-1}: the
// previous row's point and epsilon, or for a wave's first row the ones
// before it (for the window's first row, the history row x_{t-1} that the
// batch evaluated first).
template <int NW, int R, int VEC, bool NOISE, bool DPM>
__global__ __launch_bounds__(NW * 64) void k_picard_scan(
    const LoopState* __restrict__ st, float* ring, const float* __restrict__ eps,
    const float* __restrict__ noise, const float* __restrict__ Atab,
    const float* __restrict__ Btab, const float* __restrict__ Rtab,
    const float* __restrict__ Stab, int p, int batch, int64_t D, float* __restrict__ partials,
    FinalizeArgs fin, int fuse_finalize, int cpb, const float* __restrict__ eps2) {
    typedef typename Cols<VEC>::type V;
    const LoopState cur = *st;
    const int pe = cur.p_eff;
    if (pe <= 0) return;
    const int t = cur.t, f = cur.f;
    // the wave index is uniform: keep it (and every row index derived from
    // it) in scalar registers
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int b = blockIdx.y, blk = blockIdx.x, nblk = gridDim.x;
    // lane l covers columns [blk cpb + l VEC, + VEC) of the block's cpb (D and
    // cpb are multiples of VEC)
    const int64_t d = (int64_t)blk * cpb + (int64_t)lane * VEC;
    const bool valid = lane * VEC < cpb && d < D;
    const int64_t slotsz = (int64_t)batch * D;
    const int64_t col = (int64_t)b * D + (valid ? d : 0);
    const int P1 = fin.ring_slots;
    // DPM-Solver: eps row 0 holds the point before the window (once t >= 1)
    const int hist = DPM ? cur.nrows - pe : 0;
    const int ch = (pe + NW - 1) / NW;
    const int j0 = min(w * ch, pe), j1 = min(j0 + ch, pe);
    const int nr = j1 - j0;

    // a single-block grid finalizes the iteration itself, from LDS: its
    // tolerances and the timesteps of the next window are fetched now, with
    // the window's data
    __shared__ int s_mt[2 * kMaxWindow], s_mt2[2 * kMaxWindow];
    __shared__ float s_err[kMaxWindow];
    float ftol = 0.f;
    int mt_i = 0, mt2_i = 0;   // stored to LDS once the window's loads have arrived
    const bool has_mt = fuse_finalize && (int)threadIdx.x < 2 * p && t + (int)threadIdx.x < fin.T;
    if (fuse_finalize) {
        const int i = threadIdx.x;
        if (i >= 1 && i < pe) ftol = offset_tol(fin, t, i);
        if (has_mt) {
            mt_i = fin.model_t[t + i];
            if (fin.nrow2) mt2_i = fin.model_t_next[t + i];
        }
    }

    // wave totals and first old points, then (after a barrier) the
    // per-row squared differences of every lane
    __shared__ union {
        struct {
            V tot[2][NW][64];
            V first[NW][64];
        } x;
        float d2[NW * R][65];
    } sh;

    // ---- every read of this block's ring columns is consumed before the
    // first barrier; the writes all come after it (the ring slots overlap).
    const V anchor = *reinterpret_cast<const V*>(ring + (int64_t)(t % P1) * slotsz + col);
    const int slot_f = f % P1;
    const int jt = min(j0 + (lane < R ? lane : R - 1), pe - 1);   // lane r: row j0 + r
    const float ta = Atab[t + jt], tb = Btab[t + jt];
    float tr = 0.f, ts = 0.f;
    V xp = V(0.f), ep = V(0.f);   // DPM-Solver: x and eps of the step before row j0
    if constexpr (DPM) {
        tr = Rtab[t + jt];
        ts = Stab[t + jt];
        const int mp = max(t + j0 - 1, 0);           // clamped (step 0 is first order)
        xp = *reinterpret_cast<const V*>(ring + (int64_t)(mp <= f ? mp % P1 : slot_f) * slotsz + col);
        ep = *reinterpret_cast<const V*>(eps + (int64_t)max(j0 - 1 + hist, 0) * slotsz + col);
    }
    V xo[R], y[R], z[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = min(j0 + r, pe - 1);            // clamped: always a window row
        const int m = t + j;
        const int sl = m <= f ? m % P1 : slot_f;      // points past f equal x_f
        xo[r] = *reinterpret_cast<const V*>(ring + (int64_t)sl * slotsz + col);
        y[r] = *reinterpret_cast<const V*>(eps + (int64_t)(j + hist) * slotsz + col);
        if (eps2 != nullptr && m + 1 < fin.T) {
            // Heun: the mean of the two evaluations, for every step but the
            // chain's last (which keeps its Euler drift)
            const V e2 = *reinterpret_cast<const V*>(eps2 + (int64_t)j * slotsz + col);
#pragma unroll
            for (int c = 0; c < VEC; ++c)
                col_at<VEC>(y[r], c) = __fmul_rn(__fadd_rn(col_at<VEC>(y[r], c), col_at<VEC>(e2, c)), 0.5f);
        }
        if constexpr (NOISE) z[r] = *reinterpret_cast<const V*>(noise + (int64_t)m * slotsz + col);
        else z[r] = V(0.f);
    }
    // drifts replace eps in y; rows past the wave's range count as zero
    V acc_y = V(0.f), acc_z = V(0.f);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float ca = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ta), r));
        const float cb = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, tb), r));
        const bool in = r < nr;
        float cr = 0.f, cs = 0.f;
        if constexpr (DPM) {
            cr = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, tr), r));
            cs = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ts), r));
        }
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            const float e = col_at<VEC>(y[r], c);
            float v = drift(ca, col_at<VEC>(xo[r], c), cb, e);
            if constexpr (DPM) {
                // second-order steps add R x_{m-1} + S eps_{m-1}, in that order
                const float v2 = __fadd_rn(__fadd_rn(v, __fmul_rn(cr, col_at<VEC>(xp, c))),
                                           __fmul_rn(cs, col_at<VEC>(ep, c)));
                v = cr != 0.f ? v2 : v;
                col_at<VEC>(xp, c) = col_at<VEC>(xo[r], c);
                col_at<VEC>(ep, c) = e;
            }
            col_at<VEC>(y[r], c) = in ? v : 0.f;
            if (!in) col_at<VEC>(z[r], c) = 0.f;
            col_at<VEC>(acc_y, c) = __fadd_rn(col_at<VEC>(acc_y, c), col_at<VEC>(y[r], c));
            col_at<VEC>(acc_z, c) = __fadd_rn(col_at<VEC>(acc_z, c), col_at<VEC>(z[r], c));
        }
    }
    sh.x.tot[0][w][lane] = acc_y;
    sh.x.tot[1][w][lane] = acc_z;
    sh.x.first[w][lane] = xo[0];   // x^k_{t+j0}: the previous wave's old point past its range
    if (has_mt) {
        s_mt[threadIdx.x] = mt_i;
        s_mt2[threadIdx.x] = mt2_i;
    }
    // every ring value this wave read has been consumed above, so the ring
    // writes after the next barrier cannot overtake a read
    lds_barrier();
    V py = V(0.f), pz = V(0.f);
    for (int v = 0; v < w; ++v) {
        const V a = sh.x.tot[0][v][lane], c2 = sh.x.tot[1][v][lane];
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            col_at<VEC>(py, c) = __fadd_rn(col_at<VEC>(py, c), col_at<VEC>(a, c));
            col_at<VEC>(pz, c) = __fadd_rn(col_at<VEC>(pz, c), col_at<VEC>(c2, c));
        }
    }
    const V next_old = (w + 1 < NW) ? sh.x.first[w + 1][lane] : V(0.f);
    lds_barrier();

    // ---- new points, their squared differences, and the writes
    V sy = V(0.f), sz = V(0.f);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = j0 + r;
        const bool in = r < nr;
        // error of window offset o = j + 1: x^{k+1}_{t+j+1} against x^k_{t+j+1}
        const V xold = (r + 1 < R && r + 1 < nr) ? xo[r + 1 < R ? r + 1 : r] : next_old;
        V xn;
        float acc = 0.f;
#pragma unroll
        for (int c = 0; c < VEC; ++c) {
            col_at<VEC>(sy, c) = __fadd_rn(col_at<VEC>(sy, c), col_at<VEC>(y[r], c));
            col_at<VEC>(sz, c) = __fadd_rn(col_at<VEC>(sz, c), col_at<VEC>(z[r], c));
            const float v = __fadd_rn(
                __fadd_rn(col_at<VEC>(anchor, c), __fadd_rn(col_at<VEC>(py, c), col_at<VEC>(sy, c))),
                __fadd_rn(col_at<VEC>(pz, c), col_at<VEC>(sz, c)));
            col_at<VEC>(xn, c) = v;
            if (j + 1 < pe) {
                const float dl = __fsub_rn(v, col_at<VEC>(xold, c));
                acc += dl * dl;
            } else {
                acc += isfinite(v) ? 0.f : 1.f;     // last row: count non-finite points
            }
        }
        if (in && valid) *reinterpret_cast<V*>(ring + (int64_t)((t + j + 1) % P1) * slotsz + col) = xn;
        sh.d2[w * R + r][lane] = (in && valid) ? acc : 0.f;
    }
    lds_barrier();
    // row q of the NW * R (wave, row) pairs is summed by 64 / R threads
    constexpr int TPR = 64 / R;
    const int q = threadIdx.x / TPR, part = threadIdx.x % TPR;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 64 / TPR; ++i) s += sh.d2[q][part + TPR * i];
    s = group_sum<TPR>(s);
    const int qw = q / R, qr = q % R;
    const int q0 = min(qw * ch, pe), nq = min(q0 + ch, pe) - q0;
    if (!fuse_finalize) {
        if (part == 0 && qr < nq) {
            const int jq = q0 + qr;
            partials[((int64_t)b * p + (jq + 1 < pe ? jq + 1 : 0)) * nblk + blk] = s;
        }
        return;     // the finalize step follows as its own launch
    }
    // one block, one sample: the sums are the errors' numerators; the stride
    // test and the slide follow here (the same arithmetic as the separate
    // finalize step, whose sum over one partial is that partial)
    if (part == 0 && qr < nq) {
        const int jq = q0 + qr;
        s_err[jq + 1 < pe ? jq + 1 : 0] = s;
    }
    lds_barrier();
    // thread o tests offset o; each wave records its first failing offset
    __shared__ int s_wfail[NW], s_wbad[NW];
    {
        const int o = threadIdx.x;
        bool fails = false, bad = false;
        if (o == 0) {
            bad = s_err[0] != 0.f;
        } else if (o < pe) {
            const float err = s_err[o] / fin.err_div;
            bad = !isfinite(err);
            fails = !(err <= ftol);
        }
        const uint64_t fm = __ballot(fails), bm = __ballot(bad);
        if (lane == 0) {
            s_wfail[w] = fm ? w * 64 + __ffsll((unsigned long long)fm) - 1 : pe;
            s_wbad[w] = bm != 0;
        }
    }
    lds_barrier();
    int stride = pe, bad = 0;
#pragma unroll
    for (int v = 0; v < NW; ++v) {
        stride = min(stride, s_wfail[v]);
        bad |= s_wbad[v];
    }
    finalize_apply(fin, stride, bad, cur, s_mt, fin.nrow2 ? s_mt2 : nullptr);
}


// Heun's method, sequential side: the Euler prediction of one step, and the
// averaged epsilon (both as in the window kernels above).
__global__ __launch_bounds__(256) void k_seq_heun_predict(const float* __restrict__ x,
                                                          const float* __restrict__ eps, float A,
                                                          float B, int64_t n,
                                                          float* __restrict__ xt) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    xt[i] = __fadd_rn(x[i], drift(A, x[i], B, eps[i]));
}

__global__ __launch_bounds__(256) void k_seq_heun_combine(float* __restrict__ eps,
                                                          const float* __restrict__ eps2,
                                                          int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    eps[i] = __fmul_rn(__fadd_rn(eps[i], eps2[i]), 0.5f);
}

// DPM-Solver, sequential side: x <- x + (((P x + Q eps) + R xp) + S ep) on a
// second-order step (else the first-order drift), then (xp, ep) <- (x, eps).
__global__ __launch_bounds__(256) void k_seq_step_dpm(float* __restrict__ x,
                                                      const float* __restrict__ eps,
                                                      float* __restrict__ xp,
                                                      float* __restrict__ ep, float P, float Q,
                                                      float R, float S, int second, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float xi = x[i], ei = eps[i];
    float y = drift(P, xi, Q, ei);
    if (second) y = __fadd_rn(__fadd_rn(y, __fmul_rn(R, xp[i])), __fmul_rn(S, ep[i]));
    x[i] = __fadd_rn(xi, y);
    xp[i] = xi;
    ep[i] = ei;
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

// A block covers at most 64 lanes x VEC columns.  When the grid takes more
// than one block, the columns are shared out evenly over the fewest rounds of
// one block per compute unit that the 64-lane limit allows (a multiple of VEC
// per block), so that no unit streams twice the data of another: at
// 4x96x96 and one sample, 256 blocks of 144 columns instead of 144 of 256.
int picard_scan_cols(int64_t D, int batch) {
    const int vec = scan_vec(D);
    const int64_t full = 64 * (int64_t)vec;
    const int64_t blocks = (D + full - 1) / full * batch;
    const int64_t cus = device_cus();
    // one block keeps the fused finalize; a grid under half the units gains nothing
    if (blocks <= 1 || 2 * blocks < cus) return (int)full;
    const int64_t rounds = (blocks + cus - 1) / cus;
    int64_t per = (D * batch + rounds * cus - 1) / (rounds * cus);   // columns per block
    per = (per + vec - 1) / vec * vec;
    return (int)(per < full ? per : full);
}
int picard_partial_blocks(int64_t D, int batch) {
    const int64_t cols = picard_scan_cols(D, batch);
    return (int)((D + cols - 1) / cols);
}

static unsigned stream_blocks(int64_t n) {
    const int64_t b = (n + 255) / 256;
    return (unsigned)(b < 4096 ? (b > 0 ? b : 1) : 4096);
}

void launch_heun_predict(const LoopState* st, const float* ring, const float* eps, const float* A,
                         const float* B, int p, int64_t BD, float* xt, hipStream_t s) {
    hipLaunchKernelGGL(k_heun_predict, dim3(stream_blocks((int64_t)p * BD)), dim3(256), 0, s, st,
                       ring, eps, A, B, p, BD, xt);
    PD_HIP(hipGetLastError());
}

void launch_seq_heun_predict(const float* x, const float* eps, float A, float B, int64_t n,
                             float* xt, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_seq_heun_predict, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x,
                       eps, A, B, n, xt);
    PD_HIP(hipGetLastError());
}

void launch_seq_step_dpm(float* x, const float* eps, float* xp, float* ep, float P, float Q, float R,
                         float S, bool second, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_seq_step_dpm, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x, eps, xp,
                       ep, P, Q, R, S, (int)second, n);
    PD_HIP(hipGetLastError());
}

void launch_seq_heun_combine(float* eps, const float* eps2, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_seq_heun_combine, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, eps,
                       eps2, n);
    PD_HIP(hipGetLastError());
}

template <int NW, int R, int VEC>
static bool launch_scan(const LoopState* st, float* ring, const float* eps, const float* noise,
                        const float* A, const float* B, const float* Rt, const float* St, int p,
                        int batch, int64_t D, float* partials, const FinalizeArgs& fin,
                        const float* eps2, hipStream_t s) {
    const int cpb = picard_scan_cols(D, batch);
    const dim3 grid((unsigned)picard_partial_blocks(D, batch), (unsigned)batch);
    const int fuse = grid.x * grid.y == 1;   // one block: the finalize works from LDS
    const dim3 block(NW * 64);
    if (Rt)      // DPM-Solver integrates the noise-free chain
        hipLaunchKernelGGL((k_picard_scan<NW, R, VEC, false, true>), grid, block, 0, s, st, ring, eps,
                           noise, A, B, Rt, St, p, batch, D, partials, fin, fuse, cpb, eps2);
    else if (noise)
        hipLaunchKernelGGL((k_picard_scan<NW, R, VEC, true, false>), grid, block, 0, s, st, ring, eps,
                           noise, A, B, Rt, St, p, batch, D, partials, fin, fuse, cpb, eps2);
    else
        hipLaunchKernelGGL((k_picard_scan<NW, R, VEC, false, false>), grid, block, 0, s, st, ring, eps,
                           noise, A, B, Rt, St, p, batch, D, partials, fin, fuse, cpb, eps2);
    PD_HIP(hipGetLastError());
    return fuse != 0;
}

bool launch_picard_scan(const LoopState* st, float* ring, const float* eps, const float* noise,
                        const float* A, const float* B, const float* R, const float* S, int p,
                        int batch, int64_t D, float* partials, const FinalizeArgs& fin,
                        const float* eps2, hipStream_t s) {
    if (p > kMaxWindow) fail(PD_ERR_UNSUPPORTED, "window larger than 128 points");
    if (R && noise) fail(PD_ERR_INVALID_ARG, "the multistep drift is for the noise-free chain");
    if (R && eps2) fail(PD_ERR_INVALID_ARG, "the multistep and Heun drifts do not combine");
    const bool v4 = scan_vec(D) == 4;
#define PD_SCAN(NW, RR)                                                                          \
    return v4 ? launch_scan<NW, RR, 4>(st, ring, eps, noise, A, B, R, S, p, batch, D, partials, \
                                       fin, eps2, s)                                             \
              : launch_scan<NW, RR, 1>(st, ring, eps, noise, A, B, R, S, p, batch, D, partials, \
                                       fin, eps2, s);
    if (p > 64) PD_SCAN(16, 8)
    const int ch = (p + 7) / 8;      // rows per wave at a full window, 8 waves
    if (ch <= 1) PD_SCAN(8, 1)
    if (ch <= 2) PD_SCAN(8, 2)
    if (ch <= 4) PD_SCAN(8, 4)
    PD_SCAN(8, 8)
#undef PD_SCAN
}

bool mlp_head_scan_fits(int p) { return p >= 1 && p <= kMaxWindow; }

void launch_mlp_head_scan(const HeadScanArgs& a, const FinalizeArgs& fin, hipStream_t s) {
    if (!mlp_head_scan_fits(fin.p)) fail(PD_ERR_UNSUPPORTED, "window larger than the fused head takes");
    if ((a.l4.K % 4) != 0) fail(PD_ERR_UNSUPPORTED, "mlp layer sizes must be multiples of 4");
    if (a.n_slabs != (int)((a.D + 15) / 16) || fin.history || fin.nrow2)
        fail(PD_ERR_INVALID_ARG, "fused head: slab count or drift kind mismatch");
    const dim3 grid((unsigned)a.n_slabs, (unsigned)(((int64_t)fin.p * a.batch + 15) / 16));
    if (a.noise)
        hipLaunchKernelGGL(k_mlp_head_scan<true>, grid, dim3(kLinWaves * 64), 0, s, a, fin);
    else
        hipLaunchKernelGGL(k_mlp_head_scan<false>, grid, dim3(kLinWaves * 64), 0, s, a, fin);
    PD_HIP(hipGetLastError());
}

void launch_picard_finalize(const FinalizeArgs& fin, hipStream_t s) {
    hipLaunchKernelGGL(k_picard_finalize, dim3(1), dim3(1024), 0, s, fin,
                       picard_partial_blocks(fin.D, fin.batch));
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
