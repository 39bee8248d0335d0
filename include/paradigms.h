/*
 * paradigms.h -- C ABI of the MI355X (gfx950) ParaDiGMS sampler.
 *
 * ParaDiGMS (Shih, Belkhale, Ermon, Sadigh, Anari: "Parallel Sampling of
 * Diffusion Models") samples a diffusion model by Picard iteration over a
 * sliding window of the denoising trajectory (Sec. 3, Algorithm 1): the
 * drifts of the p window points are evaluated as one batch, the window is
 * rebuilt from its left end plus running sums of drift and pre-drawn noise
 * (the discretised Picard rule of Sec. 3), each point's error is checked
 * against tau^2 sigma^2 (Sec. 3.1, the relaxed tolerance), and the window
 * slides past the converged prefix.
 *
 * Time runs forward along the reverse process: reverse step i in [0, T)
 * takes x_i to x_{i+1}; x_0 ~ N(0, I) is the prior point and x_T the sample.
 *
 * Conventions for every entry point
 *  - Return a pd_status; nothing throws or aborts across the ABI.  On error
 *    pd_last_error() describes it (thread-local string owned by the library,
 *    valid until the next call on the same thread).
 *  - Arguments are validated on the host before any device work, so invalid
 *    arguments give PD_ERR_INVALID_ARG also on a machine without a GPU.
 *  - "device" pointers are HIP device memory of the current device; "host"
 *    pointers are ordinary host memory.  The caller owns every pointer it
 *    passes; the library never frees them and keeps none after returning.
 *  - `stream` is a hipStream_t (NULL = the default stream).  pd_denoiser_forward
 *    and pd_normals only enqueue work; the samplers enqueue and then
 *    synchronise `stream` before returning.
 *  - Handles (pd_schedule, pd_denoiser) are immutable after creation and may
 *    be shared between threads.  A pd_workspace is owned by one caller at a
 *    time: two calls that use the same workspace concurrently race.
 *  - Layout of a sample: float32, row-major over sample_shape; a batch of
 *    samples is [batch][prod(sample_shape)].
 */
#ifndef PARADIGMS_H
#define PARADIGMS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t pd_status;
#define PD_OK 0
#define PD_ERR_INVALID_ARG 1   /* an argument is out of range or inconsistent      */
#define PD_ERR_OOM 2           /* device or host allocation failed                  */
#define PD_ERR_DEVICE 3        /* no usable GPU, or a HIP call failed               */
#define PD_ERR_NUMERIC 4       /* a trajectory point or error became non-finite     */
#define PD_ERR_UNSUPPORTED 5   /* a valid request the library does not implement     */

/* Last error message of the calling thread ("" if none). */
const char* pd_last_error(void);
/* Library version string, e.g. "paradigms-gfx950 0.1". */
const char* pd_version(void);

/* ------------------------------------------------------------------ schedule
 * Noise schedule and the per-step drift coefficients (Sec. 2, the DDPM
 * inference model with predicted mean and time-dependent variance sigma_t^2;
 * DDIM of Song et al. as a step-reducing sampler, Sec. 2.1).  The drift that
 * Algorithm 1 consumes, "p_theta(x) - x", is y_i = A_i x + B_i eps(x, n_i),
 * where eps is the network's noise prediction and n_i its timestep.
 *
 *   linear beta_n = beta_start + n (beta_end - beta_start)/(T_train - 1),
 *   abar_n = prod_{m<=n} (1 - beta_m).
 *   PD_DDPM (T == T_train): n_i = T-1-i, A_i = 1/sqrt(alpha_n) - 1,
 *     B_i = -beta_n / (sqrt(alpha_n) sqrt(1-abar_n)),
 *     noise and tolerance variance sigma_i^2 = beta_n (1-abar_{n-1})/(1-abar_n)
 *     (zero for the last step).
 *   PD_DDIM (T_train % T == 0, c = T_train/T): n_i = (T-1-i) c, a' = abar_{n_i-c}
 *     (1 past the end), s2 = eta^2 (1-a')/(1-abar_n) (1-abar_n/a'),
 *     A_i = sqrt(a'/abar_n) - 1, B_i = sqrt(1-a'-s2) - sqrt(a'(1-abar_n)/abar_n),
 *     noise variance s2, tolerance variance = the eta = 1 value (the paper
 *     keeps the tolerance of ODE samplers relative to the variance of the
 *     corresponding DDPM SDE, footnote in Sec. 3.1).
 *   PD_DDIM_HEUN: the PD_DDIM chain with eta = 0 (required), integrated with
 *     Heun's method instead of its Euler step (Sec. 3.3: any solver can supply
 *     the drift of Algorithm 1).  With the DDIM step as the Euler
 *     prediction x~ = x + (A_i x + B_i eps(x, n_i)), the drift of every step
 *     but the last is y_i = A_i x + (B_i / 2) (eps(x, n_i) + eps(x~, n_{i+1}));
 *     the last step (to abar = 1, no network timestep) keeps the DDIM drift.
 *     Two network evaluations per step, one for the last.
 *   PD_DDIM_DPM2M: the PD_DDIM chain with eta = 0 (required), integrated with
 *     the second-order multistep DPM-Solver++(2M) (Sec. 3.3 combines the
 *     method with DPM-Solver; its multistep form reuses the previous step's
 *     network output).  With alpha_n = sqrt(abar_n), sigma_n = sqrt(1-abar_n),
 *     lambda_n = log(alpha_n/sigma_n), step i from n = n_i to n' = n - c with
 *     h = lambda_n' - lambda_n and r = (lambda_n - lambda_{n+c}) / h:
 *       y_i = A_i x + B_i eps(x, n_i) + R_i x_{i-1} + S_i eps(x_{i-1}, n_{i-1}),
 *       A_i = sigma_n'/sigma_n - alpha_n' expm1(-h) (1 + 1/(2r)) / alpha_n - 1,
 *       B_i = alpha_n' expm1(-h) (1 + 1/(2r)) sigma_n / alpha_n,
 *       R_i = alpha_n' expm1(-h) / (2r alpha_{n+c}),  S_i = -R_i sigma_{n+c},
 *     summed as ((A x + B eps) + R x_{i-1}) + S eps_{i-1}, for 1 <= i <= T-2;
 *     the first step (no previous one) and the last (to abar = 1) keep the
 *     DDIM drift (R = S = 0).  Picard evaluates the window's points plus
 *     x_{t-1} (once t >= 1), so one network evaluation more per iteration.
 * Tables are computed in double precision and rounded once to float.
 * tol_index_offset selects which variance the stride test of Algorithm 1
 * uses for the point x_{t+j}: 0 = sigma^2_{t+j} (default), -1 = sigma^2_{t+j-1}.
 * stop_rule selects the stride test's error and threshold (see
 * pd_sample_picard): PD_STOP_RELAXED, the relaxed tolerance of Sec. 3.1,
 * (1/D) |x^{k+1} - x^k|^2 <= tau^2 sigma^2; or PD_STOP_PROP2, Prop. 2's
 * total-variation rule |x^{k+1} - x^k|^2 <= 4 eps^2 sigma^2 / T^2, which
 * bounds the total-variation distance of the sample from the sequential
 * sampler's distribution by eps (given a linear convergence rate with factor
 * at least 2).  For one point the two rules agree when tau = 2 eps / (T sqrt D).
 */
#define PD_DDPM 0
#define PD_DDIM 1
#define PD_DDIM_HEUN 2
#define PD_DDIM_DPM2M 3
#define PD_STOP_RELAXED 0
#define PD_STOP_PROP2 1

typedef struct pd_schedule_desc {
    int32_t kind;              /* PD_DDPM, PD_DDIM, PD_DDIM_HEUN or PD_DDIM_DPM2M  */
    int32_t T_train;           /* length of the training chain, >= 2              */
    int32_t T;                 /* sampling steps; == T_train for DDPM             */
    int32_t tol_index_offset;  /* 0 or -1                                          */
    int32_t stop_rule;         /* PD_STOP_RELAXED (default) or PD_STOP_PROP2       */
    double beta_start;         /* 0 < beta_start <= beta_end < 1                   */
    double beta_end;
    double eta;                /* DDIM only, in [0, 1]; 0 for HEUN and DPM2M       */
} pd_schedule_desc;

typedef struct pd_schedule pd_schedule;

/* Builds the host tables.  Needs no GPU.  *out is owned by the caller and
 * released with pd_destroy_schedule.  INVALID_ARG for any range violation
 * listed in pd_schedule_desc. */
pd_status pd_init_schedule(const pd_schedule_desc* desc, pd_schedule** out);
void pd_destroy_schedule(pd_schedule* s);
/* Host copies of the length-T tables (any pointer may be NULL):
 * A, B (drift), noise_std (sqrt of the noise variance), tol_var (sigma^2 of
 * the stride test), model_t (network timestep n_i).  Also returns T. */
pd_status pd_schedule_tables(const pd_schedule* s, int32_t* T, float* A, float* B,
                             float* noise_std, float* tol_var, int32_t* model_t);
/* Host copies of the length-T multistep coefficients R (of x_{i-1}) and S (of
 * eps_{i-1}); all zero unless the kind is PD_DDIM_DPM2M.  Either pointer may
 * be NULL. */
pd_status pd_schedule_multistep_tables(const pd_schedule* s, float* R, float* S);

/* ------------------------------------------------------------------ denoiser
 * The network behind Algorithm 1's drift, as an epsilon predictor
 * eps(x, n).  The paper's trained networks are replaced by three synthetic
 * families with the shapes of its workloads:
 *  PD_MODEL_GMM2D   exact epsilon of an equal-weight mixture of isotropic
 *                   2-D Gaussians N(mu_k, s0^2 I) noised by the training
 *                   schedule: eps = sqrt(1-abar)/s^2 (x - a sum_k w_k mu_k),
 *                   a = sqrt(abar_n), s^2 = abar_n s0^2 + 1 - abar_n,
 *                   w = softmax(-|x - a mu_k|^2 / (2 s^2)).
 *                   sample_shape {2}; weights {means [K][2], sigma0 [1]}.
 *  PD_MODEL_MLP     4 layers D -> W -> W -> W -> D with exact GELU:
 *                   h1 = GELU(W1 x + b1 + e_n), h2 = GELU(W2 h1 + b2),
 *                   h3 = GELU(W3 h2 + b3), eps = W4 h3 + b4.
 *  PD_MODEL_CONV1X1 the same four layers applied to every pixel's channel
 *                   vector of a [C][H][W] sample, with SiLU activations
 *                   (a stack of 1x1 convolutions).  Built for C = 4 and
 *                   W in {32, 64, 96, 128, 320}; other shapes return
 *                   PD_ERR_UNSUPPORTED.
 *  e_n: sinusoidal embedding of width W, sin(n f_k) for k < W/2 and
 *  cos(n f_{k-W/2}) after, f_k = exp(-ln(1e4) k/(W/2)).
 *  Classifier-free guidance (cond_dim > 0, conv1x1 only): the conditional
 *  branch adds Wc c to the first-layer shift, and
 *  eps = eps_u + guidance (eps_c - eps_u) (the paper applies ParaDiGMS with
 *  guidance scale 7.5, Sec. 4.2).
 * weights: host float32 arrays in this order, (out, in) row-major:
 *  GMM2D: means [K*2], sigma0 [1]
 *  MLP / CONV1X1: W1 [W][Din], b1 [W], W2 [W][W], b2, W3 [W][W], b3,
 *                 W4 [Dout][W], b4 [Dout]  (+ Wc [W][cond_dim], c [cond_dim])
 *  with Din = Dout = D (MLP) or C (CONV1X1).
 * dtype PD_F32 computes the network to float32 accuracy: for conv1x1 the
 * matmuls of layers 2, 3 and 4 run on the fp16 matrix cores (layer 1 on the
 * fp32 ones).  Each weight is split into its nearest fp16 value and a
 * 2^11-scaled fp16 remainder, each activation likewise after a power-of-two
 * scale per tile of 16 pixels and layer, and three part products per
 * multiply-add leave an error of about one float32 rounding.  A conv1x1 weight of magnitude 65504 or more makes creation fail
 * with PD_ERR_UNSUPPORTED; non-finite activations propagate as in float32.
 * dtype PD_BF16 (conv1x1 only) rounds every matmul operand to bfloat16
 * (round to nearest even) and accumulates in float32.
 * The training schedule `train` supplies abar (GMM) and T_train (the range
 * of n).  Creation uploads the weights to the current device.
 */
#define PD_MODEL_GMM2D 0
#define PD_MODEL_MLP 1
#define PD_MODEL_CONV1X1 2
#define PD_F32 0
#define PD_BF16 1

typedef struct pd_model_desc {
    int32_t kind;          /* PD_MODEL_*                                  */
    int32_t dtype;         /* PD_F32 or PD_BF16                           */
    int32_t width;         /* hidden width W (mlp, conv1x1); even          */
    int32_t cond_dim;      /* 0 = unconditional                           */
    int32_t n_components;  /* GMM2D: K >= 1                               */
    float guidance;        /* used when cond_dim > 0                       */
} pd_model_desc;

typedef struct pd_denoiser pd_denoiser;

pd_status pd_denoiser_create(const pd_model_desc* desc, const int64_t* sample_shape,
                             int32_t ndim, const float* const* weights, int32_t n_weights,
                             const pd_schedule* train, pd_denoiser** out);
void pd_denoiser_destroy(pd_denoiser* d);

/* eps[m] = eps(x[m], model_t[m]) for m in [0, M) (the network evaluations of
 * Algorithm 1's drift step).  x, eps: device float [M][D]; model_t: device
 * int32 [M], each in [0, T_train); a value outside that range is clamped to
 * it (the network's tables hold only those timesteps).  Enqueued on `stream` of the denoiser's
 * device; x and eps must not overlap.  M = 0 is a no-op.  Allocates nothing:
 * the MLP's hidden activations go through scratch the denoiser allocated at
 * creation (in chunks of 1024 rows), and calls on several threads or streams
 * are ordered on the device so that they never share it at once. */
pd_status pd_denoiser_forward(const pd_denoiser* d, const float* x, const int32_t* model_t,
                              int64_t M, float* eps, void* stream);

/* The same network evaluations as pd_denoiser_forward, for callers that
 * cannot allocate or synchronise anything (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): no allocation, no
 * event or lock; the launches on `stream` are all it does.  The MLP's hidden
 * activations (2 * width floats per row) go to a static device array of
 * 2^20 floats (4 MiB) that each GPU holds until the process ends, so for the
 * MLP M * 2 * width <= 2^20 (M <= 512 at width 1024); larger M returns
 * PD_ERR_INVALID_ARG.  The mixture and conv1x1 models use no scratch and take
 * any M.  Every call on one GPU shares that array: calls whose work overlaps
 * on the device (other streams, or host threads) race and give undefined
 * results; calls ordered on one stream are safe.  Each layer overwrites its
 * part before reading it, so nothing needs clearing between calls. */
pd_status pd_denoiser_forward_static(const pd_denoiser* d, const float* x,
                                     const int32_t* model_t, int64_t M, float* eps,
                                     void* stream);

/* ------------------------------------------------------------------ noise
 * The up-front draws of Algorithm 1 (prior point and every step's noise).
 * Philox4x32-10 (Salmon et al., SC'11): key = (seed mod 2^32, seed div 2^32),
 * counter = (q mod 2^32, q div 2^32, rng_stream, 0) for block q, whose four
 * words r0..r3 give out[4q..4q+3] by Box-Muller in double precision on
 * u = (r + 0.5) 2^-32: sqrt(-2 ln u0) (cos, sin)(2 pi u1), then the same on
 * (u2, u3), each rounded once to float.  rng_stream 0 holds the prior point
 * (index b*D + d) and rng_stream 1 the unscaled step noise (index
 * (i*B + b)*D + d).  out: device float [count].  Enqueued on `stream`. */
pd_status pd_normals(uint64_t seed, uint32_t rng_stream, int64_t count, float* out, void* stream);

/* ------------------------------------------------------------------ sampling */
typedef struct pd_sample_stats {
    int32_t iters;             /* K: sampler iterations (sequential: T)               */
    int32_t trace_cap;         /* capacity of stride_trace (in)                        */
    int64_t evals_per_sample;  /* network evaluations per sample, the paper's "model
                                  evaluations": the sum of window sizes (Heun: two
                                  per window point, one for the last step;
                                  DPM2M: plus x_{t-1} once t >= 1)                */
    int64_t network_rows;      /* evals_per_sample * batch * (2 with guidance)         */
    int32_t* stride_trace;     /* optional host array: stride of each iteration        */
    int32_t time_kernels;      /* in: nonzero = bracket every denoiser, update and     */
                               /*     finalize launch with HIP events on `stream`      */
    int32_t denoiser_launches; /* out (with time_kernels): denoiser calls timed        */
    int32_t update_launches;   /* out: Picard update (scan) or sequential step launches */
    int32_t finalize_launches; /* out: stride/slide launches (Picard only)             */
    double denoiser_ms;        /* out: summed event time of the denoiser calls         */
    double update_ms;          /* out: summed event time of the update launches        */
    double finalize_ms;        /* out: summed event time of the finalize launches      */
} pd_sample_stats;
/* With the MLP denoiser and the Euler drift (PD_DDPM, PD_DDIM) ParaDiGMS runs
 * the network's last layer inside the update launch, whose epilogue is the
 * Picard update, error and stride step: denoiser_ms then times the first three
 * layers, update_ms that fused launch, and finalize_launches is 0.  With the
 * 2-D mixture, when the sample's loop state fits in one workgroup, the whole
 * loop (for Picard sampling also the up-front draws) is one launch:
 * update_launches is 1, update_ms times it, and the denoiser and finalize
 * counts are 0. */

typedef struct pd_workspace pd_workspace;

/* Buffers for sampling with window p and batch size `batch` on the current
 * device: the window ring of p+1 points (p+2 for PD_DDIM_DPM2M, which also
 * keeps x_{t-1}), the noise of all T steps, the drift batch and the loop
 * state, plus mapped pinned host memory that the kernels write the loop
 * state and the stride of every iteration into (so the host reads them
 * without copies).  Lets repeated calls avoid allocation. */
pd_status pd_workspace_create(const pd_schedule* s, const pd_denoiser* d, int32_t p,
                              int32_t batch, pd_workspace** out);
void pd_workspace_destroy(pd_workspace* w);

/* Sequential sampling, x_{i+1} = x_i + y_i + z_i for i in [0, T) (Sec. 3,
 * sequential sampling as nested evaluation of h_i).  x_out: device float
 * [batch][D].  ws may be NULL (allocated for the call) or a workspace made
 * for the same schedule, denoiser and batch with any p >= 1.  The same
 * noise_seed draws the same x_0 and z_i in both samplers. */
pd_status pd_sample_sequential(const pd_schedule* s, const pd_denoiser* d, uint64_t noise_seed,
                               int32_t batch, const int64_t* sample_shape, int32_t ndim,
                               float* x_out, pd_sample_stats* stats, pd_workspace* ws,
                               void* stream);

/* ParaDiGMS sampling, Algorithm 1, with window p (clamped to T, at most 128)
 * and tolerance tau (>= 0; +inf accepts every point whose sigma^2 > 0).  The
 * stride test fails offset j in [1, p) when, for any sample b of the batch,
 * not (e_b <= c sigma^2), with the product taken as 0 when sigma^2 = 0 and
 *   PD_STOP_RELAXED: e_b = (1/D) |x^{k+1}_{t+j} - x^k_{t+j}|^2, c = tau^2
 *                    (float product);
 *   PD_STOP_PROP2:   e_b = |x^{k+1}_{t+j} - x^k_{t+j}|^2, c = 4 tau^2 / T^2
 *                    formed in double from the float tau and rounded once
 *                    to float; tau is Prop. 2's total-variation bound eps.
 * The sums of squares are float32.  Returns PD_ERR_NUMERIC (with x_out
 * unspecified) if a point or error becomes non-finite.  x_out: device float
 * [batch][D], also written between batches of iterations (only its content
 * on return is the sample); ws as for pd_sample_sequential (its p must be
 * >= the clamped p).  PD_ERR_UNSUPPORTED for a clamped p above 128. */
pd_status pd_sample_picard(const pd_schedule* s, const pd_denoiser* d, int32_t p, float tau,
                           uint64_t noise_seed, int32_t batch, const int64_t* sample_shape,
                           int32_t ndim, float* x_out, pd_sample_stats* stats, pd_workspace* ws,
                           void* stream);

#ifdef __cplusplus
}
#endif
#endif /* PARADIGMS_H */
