// Internal declarations shared by the host runtime and the HIP kernels of
// the gfx950 ParaDiGMS library.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "paradigms.h"

namespace pd {

// ---------------------------------------------------------------- errors
struct Error {
    pd_status code;
    std::string msg;
};
[[noreturn]] void fail(pd_status code, const std::string& msg);
void hip_check(hipError_t e, const char* what);
#define PD_HIP(call) ::pd::hip_check((call), #call)

// compute units of the first device the library ran on (256 on MI355X)
int device_cus();

// ---------------------------------------------------------------- rows
// Where the rows of one denoiser batch live.  Rows come in groups of `group`
// consecutive rows (the samples of a batch at one trajectory point); group g
// is read from base + slot[g] * slot_stride (slot == nullptr: slot[g] = g) and
// row (g, b) from there + b * D.  n[g] is the network timestep of group g.
// The number of groups to process is *active (device) or max_groups.
struct RowSrc {
    const float* base;
    const int32_t* slot;
    int64_t slot_stride;
    int32_t group;
    int32_t max_groups;
    const int32_t* n;
    const int32_t* active;
    int32_t n_max;          // T_train - 1: the last timestep the network's tables hold
};
// Network timestep of row group g, clamped into the tables' range (a timestep
// outside [0, T_train) from a caller gives the nearest end's network, never a
// read past the tables).
__device__ inline int row_timestep(const RowSrc& s, int64_t g) {
    const int n = s.n[g];
    return n < 0 ? 0 : (n > s.n_max ? s.n_max : n);
}

// Loop state of one Picard run, in device memory.
struct LoopState {
    int32_t t;       // window start
    int32_t k;       // iterations done
    int32_t f;       // frontier: highest trajectory index holding a computed point
    int32_t p_eff;   // size of the current window; 0 once t >= T or after an error
    int32_t status;  // PD_OK or PD_ERR_NUMERIC
    int32_t first_stride;  // stride of iteration 0 (the window of copies of x_0)
    int32_t nrows;   // rows of the next denoiser batch: p_eff, plus one history
                     // row (the point before the window) for the multistep drift
    int64_t evals;   // network evaluations per sample
};
// The host reads the loop state from a copy in mapped, coherent pinned host
// memory that the kernels write as they change it (no copy launch per batch).
__device__ inline void mirror_state(const LoopState& v, LoopState* host) {
    if (!host) return;
    host->t = v.t;
    host->k = v.k;
    host->f = v.f;
    host->p_eff = v.p_eff;
    host->status = v.status;
    host->first_stride = v.first_stride;
    host->nrows = v.nrows;
    host->evals = v.evals;
    __threadfence_system();
}

// The start of a Picard run: the loop state and the first window's row
// descriptors, every window point a copy of x_0 (slot 0).  model_t_next and
// nrow2: Heun only (nullptr otherwise), the network timestep of each window
// row's next step and its per-window copy.  Run by the threads of one block.
struct PicardInit {
    LoopState* st;
    int32_t* slot;
    int32_t* nrow;
    const int32_t* model_t;
    const int32_t* model_t_next;
    int32_t* nrow2;
    int32_t T, p;
};
__device__ inline void picard_init_body(const PicardInit& a) {
    const int pe = a.p < a.T ? a.p : a.T;
    if (threadIdx.x == 0) {
        a.st->t = 0;
        a.st->k = 0;
        a.st->f = 0;
        a.st->p_eff = pe;
        a.st->status = PD_OK;
        a.st->first_stride = 0;
        a.st->nrows = pe;
        a.st->evals = 0;
    }
    for (int j = threadIdx.x; j < pe; j += blockDim.x) {
        a.slot[j] = 0;
        a.nrow[j] = a.model_t[j];
        if (a.nrow2) a.nrow2[j] = a.model_t_next[j];
    }
}

// ---------------------------------------------------------------- kernels
// rng.hip
void launch_normals(uint64_t seed, uint32_t rng_stream, int64_t count, const float* scale,
                    int64_t per_scale, float* out, hipStream_t s);
// A sample's up-front draws in one launch: the prior x_0 (counter stream 0, BD
// values into x0) and, when noise is given, every step's noise (stream 1,
// noise_count values, value i scaled by scale[i / per_scale]); the values are
// those of launch_normals with the same streams.  When init is given, the
// first block also starts the Picard loop (picard_init_body).
void launch_sample_setup(uint64_t seed, int64_t BD, float* x0, int64_t noise_count,
                         const float* scale, int64_t per_scale, float* noise,
                         const PicardInit* init, hipStream_t s);

// gmm.hip: exact epsilon of an isotropic 2-D Gaussian mixture.
struct GmmParams {
    const float* means;   // [K][2]
    const float* a;       // [T_train] sqrt(abar_n)
    const float* inv2s2;  // [T_train] 1 / (2 s_n^2)
    const float* coef;    // [T_train] sqrt(1 - abar_n) / s_n^2
    int32_t K;
};
void launch_gmm_eps(const GmmParams& g, const RowSrc& src, float* eps, hipStream_t s);
// The whole Picard (or sequential) loop of the mixture model in one workgroup.
struct GmmLoopArgs {
    GmmParams g;
    const float* A;         // [T] drift coefficients
    const float* B;
    const float* tol_var;   // [T]
    const int32_t* model_t; // [T]
    const float* noise;     // [T][batch][2] or nullptr
    const float* x0;        // [batch][2]
    float* out;             // [batch][2]
    LoopState* st;          // final state (t, k, evals, status)
    LoopState* st_host;     // its host copy (mapped pinned memory), or nullptr
    int32_t* trace;         // [T] stride of every iteration (mapped pinned memory)
    int32_t T, p, batch, tol_offset;
    float tau2;             // threshold factor c: offset o fails when !(err <= c sigma^2)
    float err_div;          // err = (summed squared differences) / err_div
};
// LDS bytes the Picard loop needs at least (noise read per window from HBM);
// the launcher stages all the noise in LDS when that fits in `max_lds`.
size_t gmm_loop_lds_bytes(int T, int K, int p, int batch);
void launch_gmm_picard_loop(const GmmLoopArgs& a, size_t max_lds, hipStream_t s);
void launch_gmm_sequential_loop(const GmmLoopArgs& a, hipStream_t s);

// mlp.hip: y = act(x W^T + bias [+ shift[n_row]]) with fp32 MFMA.
enum Act { ACT_NONE = 0, ACT_GELU = 1 };
struct LinearArgs {
    const float* W;       // [N][K]
    const float* bias;    // [N] (ignored when shift != nullptr)
    const float* shift;   // [T_train][N] per-timestep shift, or nullptr
    int32_t K, N;
    int32_t act;
};
// rows from `src` (gathered, first layer) or from a dense [M][K] buffer.
void launch_linear_gather(const LinearArgs& a, const RowSrc& src, int64_t D, float* y,
                          hipStream_t s);
void launch_linear_dense(const LinearArgs& a, const float* x, const RowSrc& rows, float* y,
                         hipStream_t s);

// conv.hip: per-pixel 4-layer stack with fp32 or bf16 MFMA.
// The kernels take the argument of e^-u in base 2, t = kNegLog2e u, as their
// working form of a pre-activation u: the layer-1 shifts and the biases b2, b3
// are stored multiplied by kNegLog2e (float products).
constexpr float kNegLog2e = -1.44269504f;     // -log2(e), rounded to float
struct ConvArgs {
    const void* frags;      // packed weight fragments (layout in conv.hip)
    const float* shift_u;   // [T_train][W] kNegLog2e (b1 + e_n)
    const float* shift_c;   // [T_train][W] kNegLog2e (b1 + e_n + Wc c), or nullptr
    const float* b2;        // [W] kNegLog2e b2
    const float* b3;        // [W] kNegLog2e b3
    const float* b4;
    float guidance;
    int32_t C;              // channels
    int32_t width;          // hidden width W
    int64_t P;              // pixels per sample
    int32_t bf16;
};
size_t conv_frag_bytes(int C, int width, bool bf16);
void conv_pack_weights(int C, int width, bool bf16, const float* W1, const float* W2,
                       const float* W3, const float* W4, std::vector<uint8_t>& out);
bool conv_supported(int C, int width, bool bf16);
void launch_conv1x1(const ConvArgs& a, const RowSrc& src, float* eps, hipStream_t s);

// picard.hip
// Heun on the window: Euler prediction of every row (the scan averages the
// two evaluations, launch_picard_scan's eps2).
void launch_heun_predict(const LoopState* st, const float* ring, const float* eps, const float* A,
                         const float* B, int p, int64_t BD, float* xt, hipStream_t s);
void launch_seq_heun_predict(const float* x, const float* eps, float A, float B, int64_t n,
                             float* xt, hipStream_t s);
void launch_seq_heun_combine(float* eps, const float* eps2, int64_t n, hipStream_t s);
void launch_seq_step_dpm(float* x, const float* eps, float* xp, float* ep, float P, float Q, float R,
                         float S, bool second, int64_t n, hipStream_t s);
// Blocks per sample of the scan (one column range each; the partial sums
// come per block) and the columns each covers.
int picard_partial_blocks(int64_t D, int batch);
int picard_scan_cols(int64_t D, int batch);
// Everything the stride rule and the slide need (the finalize step).
struct FinalizeArgs {
    LoopState* st;
    LoopState* st_host;         // host copy of *st (mapped pinned memory), or nullptr
    const float* partials;      // [batch][p][picard_partial_blocks(D, batch)]
    int32_t p, batch;
    int64_t D;
    int32_t T;
    const float* tol_var;
    float tau2;                 // threshold factor c: offset o fails when !(err <= c sigma^2)
    float err_div;              // err = (summed squared differences) / err_div: D or 1
    int32_t tol_offset;
    const int32_t* model_t;
    int32_t* trace;             // [T] strides (mapped pinned memory)
    int32_t* slot;
    int32_t* nrow;
    const int32_t* model_t_next;   // Heun only, else nullptr
    int32_t* nrow2;                // Heun only, else nullptr
    int32_t ring_slots;            // p + 1, or p + 2 with a history row
    int32_t history;               // 1: the next batch starts with x_{t-1} (multistep drift)
    const float* xT;               // x_T's ring slot
    float* x_out;                  // [BD]: the iteration that reaches T copies x_T here
    int64_t BD;                    // batch * D
};
// Scan + error partials of one iteration.  Returns true when the grid is a
// single block, which then also ran the finalize step (from LDS).
// R, S: the multistep (DPM-Solver) coefficients of x_{i-1} and eps_{i-1}, or
// nullptr; eps then has the history row first when st->nrows > st->p_eff.
// eps2: Heun's second evaluations [p][BD], or nullptr; every row's drift then
// takes the mean (eps + eps2) / 2 but at the chain's last step.
bool launch_picard_scan(const LoopState* st, float* ring, const float* eps, const float* noise,
                        const float* A, const float* B, const float* R, const float* S, int p,
                        int batch, int64_t D, float* partials, const FinalizeArgs& fin,
                        const float* eps2, hipStream_t s);
void launch_picard_finalize(const FinalizeArgs& fin, hipStream_t s);
// The MLP's last layer fused with the Picard update, error and finalize (Euler
// drift, no history row): one launch in place of the last layer, the scan and
// the finalize step.  partials holds [batch][p][n_slabs]; count holds
// n_slabs + 1 ints, zero between launches.
struct HeadScanArgs {
    LinearArgs l4;          // the last layer: W4 [D][W], b4, no activation
    const float* h;         // [rows][W] the third layer's output
    RowSrc rows;            // the window's rows (the layer's row count)
    const LoopState* st;
    float* ring;
    float* eps;             // [rows][D] epsilon, written and read back
    const float* noise;     // [T][batch][D] or nullptr
    const float* A;
    const float* B;
    int32_t batch;
    int64_t D;
    float* partials;
    int32_t* count;
    int32_t n_slabs;        // 16-column slabs, ceil(D / 16)
};
bool mlp_head_scan_fits(int p);
void launch_mlp_head_scan(const HeadScanArgs& a, const FinalizeArgs& fin, hipStream_t s);
void launch_seq_step(float* x, const float* eps, const float* z, float A, float B, int64_t n,
                     hipStream_t s);

}  // namespace pd
