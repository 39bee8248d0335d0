// Host runtime of the gfx950 ParaDiGMS library: the C ABI of paradigms.h,
// argument validation, schedule tables, denoiser weights on the device, the
// sampling workspace and the two sampler loops.
#include <cmath>
#include <cstring>
#include <exception>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "gmm.h"
#include "mlp.h"
#include "pd_internal.h"

namespace pd {

[[noreturn]] void fail(pd_status code, const std::string& msg) { throw Error{code, msg}; }

void hip_check(hipError_t e, const char* what) {
    if (e == hipSuccess) return;
    const pd_status code = (e == hipErrorOutOfMemory) ? PD_ERR_OOM : PD_ERR_DEVICE;
    fail(code, std::string(what) + ": " + hipGetErrorString(e));
}

namespace {

thread_local std::string g_last_error;

template <class F>
pd_status guard(F&& f) {
    try {
        f();
        g_last_error.clear();
        return PD_OK;
    } catch (const Error& e) {
        g_last_error = e.msg;
        return e.code;
    } catch (const std::bad_alloc&) {
        g_last_error = "host allocation failed";
        return PD_ERR_OOM;
    } catch (const std::exception& e) {
        g_last_error = e.what();
        return PD_ERR_DEVICE;
    } catch (...) {
        g_last_error = "unknown error";
        return PD_ERR_DEVICE;
    }
}

void require(bool ok, const std::string& msg) {
    if (!ok) fail(PD_ERR_INVALID_ARG, msg);
}

// Device buffer owned by a handle.
struct DevBuf {
    void* p = nullptr;
    size_t bytes = 0;
    DevBuf() = default;
    DevBuf(const DevBuf&) = delete;
    DevBuf& operator=(const DevBuf&) = delete;
    ~DevBuf() {
        if (p) (void)hipFree(p);
    }
    void alloc(size_t n) {
        if (p) (void)hipFree(p);
        p = nullptr;
        bytes = n;
        if (n == 0) return;
        PD_HIP(hipMalloc(&p, n));
    }
    template <class T>
    void upload(const T* src, size_t count) {
        alloc(count * sizeof(T));
        if (count) PD_HIP(hipMemcpy(p, src, count * sizeof(T), hipMemcpyHostToDevice));
    }
    template <class T>
    T* as() const {
        return static_cast<T*>(p);
    }
};

int current_device() {
    int n = 0;
    const hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || n <= 0) fail(PD_ERR_DEVICE, "no HIP device is available");
    int dev = 0;
    PD_HIP(hipGetDevice(&dev));
    hipDeviceProp_t prop;
    PD_HIP(hipGetDeviceProperties(&prop, dev));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        fail(PD_ERR_DEVICE, std::string("this library is built for gfx950, device is ") +
                                prop.gcnArchName);
    return dev;
}

std::vector<double> timestep_embedding(int n, int width) {
    const int half = width / 2;
    std::vector<double> e(width);
    for (int k = 0; k < half; ++k) {
        const double freq = std::exp(-std::log(10000.0) * (double)k / (double)half);
        const double arg = (double)n * freq;
        e[k] = std::sin(arg);
        e[half + k] = std::cos(arg);
    }
    return e;
}

// Optional per-launch timing: consecutive events recorded on the sampling
// stream; elapsed times are summed per category after the final sync.
struct KernelTimer {
    bool on = false;
    hipStream_t st = nullptr;
    std::vector<hipEvent_t> ev;
    std::vector<int> cat;            // category of the interval ending at ev[i]
    double ms[3] = {0.0, 0.0, 0.0};
    int count[3] = {0, 0, 0};
    ~KernelTimer() {
        for (hipEvent_t e : ev) (void)hipEventDestroy(e);
    }
    // category < 0: start of an interval.  Consecutive intervals share their
    // boundary event, so a start mark is only needed after a gap (a host
    // synchronisation or a copy).  The events carry no system-scope fence:
    // they are read only after the stream has been synchronised.
    void mark(int category) {
        if (!on) return;
        hipEvent_t e;
        PD_HIP(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
        ev.push_back(e);
        cat.push_back(category);
        PD_HIP(hipEventRecord(e, st));
    }
    void collect() {                 // call after the stream is synchronised
        if (!on) return;
        for (size_t i = 1; i < ev.size(); ++i) {
            if (cat[i] < 0) continue;
            float t = 0.f;
            PD_HIP(hipEventElapsedTime(&t, ev[i - 1], ev[i]));
            ms[cat[i]] += t;
            count[cat[i]] += 1;
        }
    }
};
enum { CAT_DENOISER = 0, CAT_UPDATE = 1, CAT_FINALIZE = 2 };

int64_t product(const int64_t* shape, int32_t ndim) {
    int64_t D = 1;
    for (int i = 0; i < ndim; ++i) D *= shape[i];
    return D;
}

}  // namespace

int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        PD_HIP(hipGetDevice(&dev));
        PD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
        if (cus <= 0) cus = 256;
    }
    return cus;
}

}  // namespace pd

using namespace pd;

// ============================================================== schedule
struct pd_schedule {
    pd_schedule_desc desc;
    int T = 0, T_train = 0;
    std::vector<float> A, B, noise_std, tol_var;
    std::vector<int32_t> model_t;
    std::vector<int32_t> model_t_next;   // n_{i+1}; the last step repeats n_{T-1}
    std::vector<float> R, S;   // multistep coefficients of x_{i-1}, eps_{i-1} (zero: first order)
    std::vector<double> alphabar;
    bool has_noise = false;
    bool heun = false;
    bool dpm = false;          // the drift also reads the previous step (DPM-Solver++(2M))
};

static void build_tables(pd_schedule& s) {
    const pd_schedule_desc& d = s.desc;
    const int Tt = d.T_train, T = d.T;
    std::vector<double> beta(Tt), ab(Tt);
    const double step = Tt > 1 ? (d.beta_end - d.beta_start) / (double)(Tt - 1) : 0.0;
    double acc = 1.0;
    for (int n = 0; n < Tt; ++n) {
        beta[n] = d.beta_start + (double)n * step;
        acc = acc * (1.0 - beta[n]);
        ab[n] = acc;
    }
    s.T = T;
    s.T_train = Tt;
    s.alphabar = ab;
    s.A.resize(T);
    s.B.resize(T);
    s.noise_std.resize(T);
    s.tol_var.resize(T);
    s.model_t.resize(T);
    s.model_t_next.resize(T);
    s.R.assign(T, 0.f);
    s.S.assign(T, 0.f);
    s.has_noise = false;
    s.heun = d.kind == PD_DDIM_HEUN;
    s.dpm = d.kind == PD_DDIM_DPM2M;
    for (int i = 0; i < T; ++i) {
        double A, B, var, tol;
        int n;
        if (d.kind == PD_DDPM) {
            n = T - 1 - i;
            const double a = 1.0 - beta[n];
            const double ab_prev = n >= 1 ? ab[n - 1] : 1.0;
            A = 1.0 / std::sqrt(a) - 1.0;
            B = -beta[n] / (std::sqrt(a) * std::sqrt(1.0 - ab[n]));
            var = beta[n] * (1.0 - ab_prev) / (1.0 - ab[n]);
            tol = var;
        } else {
            const int c = Tt / T;
            n = (T - 1 - i) * c;
            const int npv = n - c;
            const double ap = npv >= 0 ? ab[npv] : 1.0;
            const double an = ab[n];
            const double v1 = (1.0 - ap) / (1.0 - an) * (1.0 - an / ap);
            const double s2 = d.eta * d.eta * v1;
            A = std::sqrt(ap / an) - 1.0;
            B = std::sqrt(1.0 - ap - s2) - std::sqrt(ap * (1.0 - an) / an);
            var = s2;
            tol = v1;
        }
        s.model_t[i] = n;
        s.A[i] = (float)A;
        s.B[i] = (float)B;
        s.noise_std[i] = (float)std::sqrt(var);
        s.tol_var[i] = (float)tol;
        if (var > 0.0) s.has_noise = true;
    }
    if (s.dpm) {
        // DPM-Solver++(2M) in the data-prediction form x0 = (x - sigma eps)/alpha,
        // with alpha_n = sqrt(abar_n), sigma_n = sqrt(1 - abar_n), lambda = log(alpha/sigma).
        // Step i goes from n = n_i to n - c with h = lambda(n - c) - lambda(n); the
        // previous step's data prediction (from n + c) enters through
        // r = (lambda(n) - lambda(n + c)) / h:
        //   x' = (sigma'/sigma) x - alpha' expm1(-h) ((1 + 1/(2r)) x0 - x0_prev/(2r)).
        // Written as x' - x = P x + Q eps + R x_prev + S eps_prev (A, B hold P, Q).
        // The first step has no previous one and the last (to abar = 1) is
        // taken to first order: both keep the DDIM drift.
        const int c = Tt / T;
        auto alpha = [&](int n) { return std::sqrt(ab[n]); };
        auto sigma = [&](int n) { return std::sqrt(1.0 - ab[n]); };
        auto lambda = [&](int n) { return std::log(alpha(n) / sigma(n)); };
        for (int i = 1; i + 1 < T; ++i) {
            const int n = s.model_t[i], nn = n - c, np = n + c;
            const double h = lambda(nn) - lambda(n);
            const double r = (lambda(n) - lambda(np)) / h;
            const double em = std::expm1(-h);
            const double w_cur = 1.0 + 1.0 / (2.0 * r), w_prev = 1.0 / (2.0 * r);
            s.A[i] = (float)(sigma(nn) / sigma(n) - alpha(nn) * em * w_cur / alpha(n) - 1.0);
            s.B[i] = (float)(alpha(nn) * em * w_cur * sigma(n) / alpha(n));
            const double Rc = alpha(nn) * em * w_prev / alpha(np);
            s.R[i] = (float)Rc;
            s.S[i] = (float)(-Rc * sigma(np));
        }
    }
    // the step after i; the last step has none and keeps its Euler drift, so
    // its (unused) second evaluation is pointed at a valid timestep
    for (int i = 0; i < T; ++i) s.model_t_next[i] = s.model_t[i + 1 < T ? i + 1 : i];
}

extern "C" pd_status pd_init_schedule(const pd_schedule_desc* desc, pd_schedule** out) {
    return guard([&] {
        require(desc != nullptr && out != nullptr, "desc and out must not be NULL");
        *out = nullptr;
        const pd_schedule_desc& d = *desc;
        require(d.kind == PD_DDPM || d.kind == PD_DDIM || d.kind == PD_DDIM_HEUN ||
                    d.kind == PD_DDIM_DPM2M,
                "kind must be PD_DDPM, PD_DDIM, PD_DDIM_HEUN or PD_DDIM_DPM2M");
        require(d.T_train >= 2, "T_train must be >= 2");
        require(d.T >= 1 && d.T <= d.T_train, "T must be in [1, T_train]");
        require(d.kind != PD_DDPM || d.T == d.T_train, "DDPM needs T == T_train");
        require(d.kind == PD_DDPM || d.T_train % d.T == 0, "DDIM needs T_train % T == 0");
        require(std::isfinite(d.beta_start) && std::isfinite(d.beta_end) && d.beta_start > 0.0 &&
                    d.beta_end < 1.0 && d.beta_start <= d.beta_end,
                "need 0 < beta_start <= beta_end < 1");
        require(d.kind != PD_DDIM || (d.eta >= 0.0 && d.eta <= 1.0), "eta must be in [0, 1]");
        require(d.kind != PD_DDIM_HEUN || d.eta == 0.0, "Heun integrates the eta = 0 (ODE) chain only");
        require(d.kind != PD_DDIM_DPM2M || d.eta == 0.0,
                "DPM-Solver integrates the eta = 0 (ODE) chain only");
        require(d.tol_index_offset == 0 || d.tol_index_offset == -1,
                "tol_index_offset must be 0 or -1");
        require(d.stop_rule == PD_STOP_RELAXED || d.stop_rule == PD_STOP_PROP2,
                "stop_rule must be PD_STOP_RELAXED or PD_STOP_PROP2");
        auto s = std::make_unique<pd_schedule>();
        s->desc = d;
        if (d.kind == PD_DDPM) s->desc.eta = 1.0;
        build_tables(*s);
        *out = s.release();
    });
}

extern "C" void pd_destroy_schedule(pd_schedule* s) { delete s; }

extern "C" pd_status pd_schedule_tables(const pd_schedule* s, int32_t* T, float* A, float* B,
                                        float* noise_std, float* tol_var, int32_t* model_t) {
    return guard([&] {
        require(s != nullptr, "schedule must not be NULL");
        if (T) *T = s->T;
        const size_t n = (size_t)s->T;
        if (A) std::memcpy(A, s->A.data(), n * sizeof(float));
        if (B) std::memcpy(B, s->B.data(), n * sizeof(float));
        if (noise_std) std::memcpy(noise_std, s->noise_std.data(), n * sizeof(float));
        if (tol_var) std::memcpy(tol_var, s->tol_var.data(), n * sizeof(float));
        if (model_t) std::memcpy(model_t, s->model_t.data(), n * sizeof(int32_t));
    });
}

extern "C" pd_status pd_schedule_multistep_tables(const pd_schedule* s, float* R, float* S) {
    return guard([&] {
        require(s != nullptr, "schedule must not be NULL");
        const size_t n = (size_t)s->T;
        if (R) std::memcpy(R, s->R.data(), n * sizeof(float));
        if (S) std::memcpy(S, s->S.data(), n * sizeof(float));
    });
}

extern "C" const char* pd_last_error(void) { return g_last_error.c_str(); }
extern "C" const char* pd_version(void) { return "paradigms-gfx950 0.1"; }

// ============================================================== denoiser
// pd_denoiser_forward runs the MLP's hidden layers through a scratch buffer
// the denoiser allocates once, at creation, for this many rows; larger calls
// are processed in chunks of it.
static constexpr int64_t kForwardRows = 1024;

struct pd_denoiser {
    pd_model_desc desc{};
    std::vector<int64_t> shape;
    int64_t D = 0, P = 0;
    int C = 0, T_train = 0, device = 0;
    // gmm2d
    DevBuf means, g_a, g_inv2s2, g_coef;
    // mlp
    DevBuf W[4], bias[4], shift1;
    // conv1x1
    DevBuf frags, shift_u, shift_c;
    // pd_denoiser_forward's MLP scratch (kForwardRows rows).  Calls may come
    // from several threads and streams: under fwd_mu, each call's kernels wait
    // for fwd_done, the end of the previous call's use, and record it anew.
    DevBuf fwd_scratch;
    hipEvent_t fwd_done = nullptr;
    mutable std::mutex fwd_mu;

    ~pd_denoiser() {
        if (fwd_done) (void)hipEventDestroy(fwd_done);
    }

    bool guided() const { return desc.cond_dim > 0; }

    GmmParams gmm() const {
        return GmmParams{means.as<float>(), g_a.as<float>(), g_inv2s2.as<float>(), g_coef.as<float>(),
                         desc.n_components};
    }

    size_t scratch_floats(int64_t rows) const {
        return desc.kind == PD_MODEL_MLP ? (size_t)(2 * rows * desc.width) : 0;
    }

    // MLP: the first three layers through scratch (2 * rows * width floats);
    // returns the third layer's output, the last layer's input
    const float* mlp_trunk(const RowSrc& src, float* scratch, hipStream_t s) const {
        const int Wd = desc.width;
        const int64_t rows = (int64_t)src.max_groups * src.group;
        float* h1 = scratch;
        float* h2 = scratch + rows * Wd;
        LinearArgs l1{W[0].as<float>(), nullptr, shift1.as<float>(), (int)D, Wd, ACT_GELU};
        LinearArgs l2{W[1].as<float>(), bias[1].as<float>(), nullptr, Wd, Wd, ACT_GELU};
        LinearArgs l3{W[2].as<float>(), bias[2].as<float>(), nullptr, Wd, Wd, ACT_GELU};
        launch_linear_gather(l1, src, D, h1, s);
        launch_linear_dense(l2, h1, src, h2, s);
        launch_linear_dense(l3, h2, src, h1, s);
        return h1;
    }
    // MLP: the last layer (no activation)
    LinearArgs mlp_head() const {
        return LinearArgs{W[3].as<float>(), bias[3].as<float>(), nullptr, desc.width, (int)D, ACT_NONE};
    }

    void forward(const RowSrc& src, float* eps, float* scratch, hipStream_t s) const {
        switch (desc.kind) {
            case PD_MODEL_GMM2D:
                launch_gmm_eps(gmm(), src, eps, s);
                break;
            case PD_MODEL_MLP:
                launch_linear_dense(mlp_head(), mlp_trunk(src, scratch, s), src, eps, s);
                break;
            case PD_MODEL_CONV1X1: {
                ConvArgs a{frags.p,           shift_u.as<float>(),
                           guided() ? shift_c.as<float>() : nullptr,
                           bias[1].as<float>(), bias[2].as<float>(), bias[3].as<float>(),
                           desc.guidance,     C,
                           desc.width,        P,
                           desc.dtype == PD_BF16 ? 1 : 0};
                launch_conv1x1(a, src, eps, s);
                break;
            }
            default:
                fail(PD_ERR_UNSUPPORTED, "unknown model kind");
        }
    }
};

static void create_denoiser(const pd_model_desc& m, const int64_t* shape, int32_t ndim,
                            const float* const* w, int32_t nw, const pd_schedule& train,
                            pd_denoiser& d) {
    d.desc = m;
    d.shape.assign(shape, shape + ndim);
    d.D = product(shape, ndim);
    d.T_train = train.T_train;
    const int Tt = train.T_train;
    if (m.kind == PD_MODEL_GMM2D) {
        require(ndim == 1 && shape[0] == 2, "gmm2d samples have shape {2}");
        require(m.n_components >= 1 && m.n_components <= 64, "gmm2d needs 1..64 components");
        require(m.cond_dim == 0 && m.dtype == PD_F32, "gmm2d is unconditional float32");
        require(nw == 2, "gmm2d takes 2 weight arrays (means, sigma0)");
        d.device = current_device();
        const double s0 = (double)w[1][0];
        std::vector<float> a(Tt), inv2s2(Tt), coef(Tt);
        for (int n = 0; n < Tt; ++n) {
            const double ab = train.alphabar[n];
            const double s2 = ab * (s0 * s0) + 1.0 - ab;
            a[n] = (float)std::sqrt(ab);
            inv2s2[n] = (float)(1.0 / (2.0 * s2));
            coef[n] = (float)(std::sqrt(1.0 - ab) / s2);
        }
        d.means.upload(w[0], (size_t)2 * m.n_components);
        d.g_a.upload(a.data(), a.size());
        d.g_inv2s2.upload(inv2s2.data(), inv2s2.size());
        d.g_coef.upload(coef.data(), coef.size());
        return;
    }
    require(m.kind == PD_MODEL_MLP || m.kind == PD_MODEL_CONV1X1, "unknown model kind");
    require(m.width >= 2 && m.width % 2 == 0, "width must be even and >= 2");
    require(m.cond_dim >= 0, "cond_dim must be >= 0");
    require(m.dtype == PD_F32 || m.dtype == PD_BF16, "dtype must be PD_F32 or PD_BF16");
    const int Wd = m.width;
    int Din;
    if (m.kind == PD_MODEL_MLP) {
        require(m.cond_dim == 0, "guidance is implemented for conv1x1 only");
        require(m.dtype == PD_F32, "the mlp denoiser is float32");
        require(d.D % 4 == 0 && Wd % 4 == 0, "mlp sizes must be multiples of 4");
        Din = (int)d.D;
    } else {
        require(ndim == 3, "conv1x1 samples have shape {C, H, W}");
        d.C = (int)shape[0];
        d.P = shape[1] * shape[2];
        require(d.C >= 1 && d.P >= 1, "empty conv1x1 sample shape");
        if (!conv_supported(d.C, Wd, m.dtype == PD_BF16))
            fail(PD_ERR_UNSUPPORTED, "conv1x1: this channel count / width / dtype is not built");
        Din = d.C;
    }
    const int nexp = 8 + (m.cond_dim > 0 ? 2 : 0);
    require(nw == nexp, "wrong number of weight arrays");
    for (int i = 0; i < nw; ++i) require(w[i] != nullptr, "weight array is NULL");
    if (m.cond_dim > 0) require(std::isfinite(m.guidance), "guidance must be finite");
    d.device = current_device();

    // first-layer shift b1 + e_n for every network timestep (float adds)
    std::vector<float> sh((size_t)Tt * Wd);
    for (int n = 0; n < Tt; ++n) {
        const std::vector<double> e = timestep_embedding(n, Wd);
        for (int k = 0; k < Wd; ++k) sh[(size_t)n * Wd + k] = w[1][k] + (float)e[k];
    }
    const float* W1 = w[0];
    const float* W2 = w[2];
    const float* W3 = w[4];
    const float* W4 = w[6];
    d.bias[1].upload(w[3], Wd);
    d.bias[2].upload(w[5], Wd);
    d.bias[3].upload(w[7], (size_t)Din);
    if (m.kind == PD_MODEL_MLP) {
        d.W[0].upload(W1, (size_t)Wd * Din);
        d.W[1].upload(W2, (size_t)Wd * Wd);
        d.W[2].upload(W3, (size_t)Wd * Wd);
        d.W[3].upload(W4, (size_t)Din * Wd);
        d.shift1.upload(sh.data(), sh.size());
        d.fwd_scratch.alloc(d.scratch_floats(kForwardRows) * sizeof(float));
        PD_HIP(hipEventCreateWithFlags(&d.fwd_done, hipEventDisableTiming));
        return;
    }
    std::vector<uint8_t> packed;
    conv_pack_weights(d.C, Wd, m.dtype == PD_BF16, W1, W2, W3, W4, packed);
    d.frags.upload(packed.data(), packed.size());
    // the kernels take the layer-1 shifts and the biases b2, b3 times kNegLog2e
    auto scale = [](std::vector<float> v) {
        for (float& x : v) x *= kNegLog2e;
        return v;
    };
    d.bias[1].upload(scale(std::vector<float>(w[3], w[3] + Wd)).data(), Wd);
    d.bias[2].upload(scale(std::vector<float>(w[5], w[5] + Wd)).data(), Wd);
    {
        const std::vector<float> shs = scale(sh);
        d.shift_u.upload(shs.data(), shs.size());
    }
    if (m.cond_dim > 0) {
        const float* Wc = w[8];
        const float* c = w[9];
        std::vector<float> wc(Wd);
        for (int k = 0; k < Wd; ++k) {
            double acc = 0.0;
            for (int j = 0; j < m.cond_dim; ++j) acc += (double)Wc[(size_t)k * m.cond_dim + j] * c[j];
            wc[k] = (float)acc;
        }
        std::vector<float> shc(sh.size());
        for (int n = 0; n < Tt; ++n)
            for (int k = 0; k < Wd; ++k) shc[(size_t)n * Wd + k] = sh[(size_t)n * Wd + k] + wc[k];
        shc = scale(std::move(shc));
        d.shift_c.upload(shc.data(), shc.size());
    }
}

extern "C" pd_status pd_denoiser_create(const pd_model_desc* desc, const int64_t* sample_shape,
                                        int32_t ndim, const float* const* weights,
                                        int32_t n_weights, const pd_schedule* train,
                                        pd_denoiser** out) {
    return guard([&] {
        require(desc && sample_shape && weights && train && out, "NULL argument");
        *out = nullptr;
        require(ndim >= 1 && ndim <= 8, "ndim must be in [1, 8]");
        for (int i = 0; i < ndim; ++i) require(sample_shape[i] >= 1, "sample_shape entries must be >= 1");
        require(n_weights >= 1, "no weights");
        auto d = std::make_unique<pd_denoiser>();
        create_denoiser(*desc, sample_shape, ndim, weights, n_weights, *train, *d);
        *out = d.release();
    });
}

extern "C" void pd_denoiser_destroy(pd_denoiser* d) { delete d; }

extern "C" pd_status pd_denoiser_forward(const pd_denoiser* d, const float* x,
                                         const int32_t* model_t, int64_t M, float* eps,
                                         void* stream) {
    return guard([&] {
        require(d != nullptr, "denoiser must not be NULL");
        require(M >= 0 && M <= (int64_t)1 << 30, "M out of range");
        if (M == 0) return;
        require(x && model_t && eps, "NULL device pointer");
        int dev = 0;
        PD_HIP(hipGetDevice(&dev));
        require(dev == d->device, "the denoiser lives on another device");
        const hipStream_t s = static_cast<hipStream_t>(stream);
        if (!d->scratch_floats(1)) {          // no scratch: one enqueue of the whole batch
            const RowSrc src{x, nullptr, d->D, 1, (int32_t)M, model_t, nullptr, d->T_train - 1};
            d->forward(src, eps, nullptr, s);
            return;
        }
        // MLP: chunks of kForwardRows rows through the denoiser's scratch, after
        // every earlier call's kernels that used it (a wait on an event no call
        // has recorded yet is a no-op)
        const std::lock_guard<std::mutex> lock(d->fwd_mu);
        PD_HIP(hipStreamWaitEvent(s, d->fwd_done, 0));
        for (int64_t m0 = 0; m0 < M; m0 += kForwardRows) {
            const int64_t mc = M - m0 < kForwardRows ? M - m0 : kForwardRows;
            const RowSrc src{x + m0 * d->D, nullptr, d->D, 1, (int32_t)mc, model_t + m0, nullptr,
                             d->T_train - 1};
            d->forward(src, eps + m0 * d->D, d->fwd_scratch.as<float>(), s);
        }
        PD_HIP(hipEventRecord(d->fwd_done, s));
    });
}

// ============================================================== allocation-free forward
// pd_denoiser_forward_static, for callers that cannot allocate device memory
// (code under graph capture, tight serving loops): the MLP's hidden layers
// run through this file-scope device array instead of the denoiser's scratch.
// Each GPU holds its own copy until the process ends.  In host code the name
// stands for a host-side symbol, not a device address: kernels get the
// address hipGetSymbolAddress returns for the current device.
static constexpr size_t kStaticScratchFloats = (size_t)1 << 20;   // 4 MiB
static __device__ __align__(256) float scratch[kStaticScratchFloats];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev`, which must be current; looked
// up on the first call on each device.
float* static_scratch(int dev) {
    require(dev >= 0 && dev < kMaxDevices, "device index beyond the static scratch table");
    const std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        PD_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) fail(PD_ERR_DEVICE, "hipGetSymbolAddress returned no address for the static scratch");
        g_scratch_ptr[dev] = static_cast<float*>(p);
    }
    return g_scratch_ptr[dev];
}
}  // namespace

extern "C" pd_status pd_denoiser_forward_static(const pd_denoiser* d, const float* x,
                                                const int32_t* model_t, int64_t M, float* eps,
                                                void* stream) {
    return guard([&] {
        require(d != nullptr, "denoiser must not be NULL");
        require(M >= 0 && M <= (int64_t)1 << 30, "M out of range");
        const size_t need = d->scratch_floats(M);
        if (need > kStaticScratchFloats)
            fail(PD_ERR_INVALID_ARG,
                 "M = " + std::to_string(M) + " needs " + std::to_string(need) +
                     " floats of scratch; the static scratch holds " +
                     std::to_string(kStaticScratchFloats) + " (M <= " +
                     std::to_string(kStaticScratchFloats / d->scratch_floats(1)) +
                     " at this width)");
        if (M == 0) return;
        require(x && model_t && eps, "NULL device pointer");
        int dev = 0;
        PD_HIP(hipGetDevice(&dev));
        require(dev == d->device, "the denoiser lives on another device");
        const RowSrc src{x, nullptr, d->D, 1, (int32_t)M, model_t, nullptr, d->T_train - 1};
        d->forward(src, eps, need ? static_scratch(dev) : nullptr, static_cast<hipStream_t>(stream));
    });
}

// ============================================================== noise
extern "C" pd_status pd_normals(uint64_t seed, uint32_t rng_stream, int64_t count, float* out,
                                void* stream) {
    return guard([&] {
        require(count >= 0, "count must be >= 0");
        if (count == 0) return;
        require(out != nullptr, "out must not be NULL");
        launch_normals(seed, rng_stream, count, nullptr, 1, out, static_cast<hipStream_t>(stream));
    });
}

// ============================================================== workspace
struct pd_workspace {
    int device = 0;
    const pd_schedule* s = nullptr;
    const pd_denoiser* d = nullptr;
    int p = 0, batch = 0, T = 0;
    int64_t D = 0;
    DevBuf ring, eps, noise, A, B, zstd, tolv, model_t, state, slot, nrow, partials, scratch;
    DevBuf xt, eps2, model_t_next, nrow2;   // Heun: predictions, second epsilons, n_{i+1}
    DevBuf Rt, St, xprev, eprev;            // multistep: tables; the sequential loop's last step
    DevBuf head_count;                      // fused MLP head: arrival counters per slab, + 1
    int ring_slots() const { return p + 1 + (s->dpm ? 1 : 0); }
    // mapped, coherent pinned host memory that the kernels write directly:
    // the loop state's host copy and the stride of every iteration
    LoopState* h_state = nullptr;
    LoopState* h_state_dev = nullptr;   // the device's address of h_state
    hipEvent_t batch_event = nullptr;   // before the last iteration of a batch
    int32_t* h_trace = nullptr;
    int32_t* h_trace_dev = nullptr;
    ~pd_workspace() {
        if (h_state) (void)hipHostFree(h_state);
        if (h_trace) (void)hipHostFree(h_trace);
        if (batch_event) (void)hipEventDestroy(batch_event);
    }
};

template <class T>
static void host_mapped(T** host, T** dev, size_t count) {
    PD_HIP(hipHostMalloc(reinterpret_cast<void**>(host), sizeof(T) * count,
                         hipHostMallocMapped | hipHostMallocCoherent));
    std::memset(*host, 0, sizeof(T) * count);
    PD_HIP(hipHostGetDevicePointer(reinterpret_cast<void**>(dev), *host, 0));
}

// The MLP's last layer runs as the Picard update's prologue (one launch for
// the layer, the update and the stride) when the drift is the Euler step.
static bool use_mlp_head(const pd_schedule& s, const pd_denoiser& d, int p) {
    return d.desc.kind == PD_MODEL_MLP && !s.heun && !s.dpm && mlp_head_scan_fits(p);
}
static int head_slabs(int64_t D) { return (int)((D + 15) / 16); }

static void create_workspace(const pd_schedule& s, const pd_denoiser& d, int p, int batch,
                             pd_workspace& w) {
    w.device = current_device();
    require(w.device == d.device, "the denoiser lives on another device");
    require(s.T_train == d.T_train, "schedule and denoiser disagree on T_train");
    w.s = &s;
    w.d = &d;
    w.p = p;
    w.batch = batch;
    w.T = s.T;
    w.D = d.D;
    const int64_t BD = (int64_t)batch * d.D;
    // multistep: the ring also keeps x_{t-1}, and the batch starts with it
    const int hist = s.dpm ? 1 : 0;
    w.ring.alloc(sizeof(float) * (size_t)(p + 1 + hist) * BD);
    w.eps.alloc(sizeof(float) * (size_t)(p + hist) * BD);
    if (s.has_noise) w.noise.alloc(sizeof(float) * (size_t)s.T * BD);
    w.A.upload(s.A.data(), s.T);
    w.B.upload(s.B.data(), s.T);
    w.zstd.upload(s.noise_std.data(), s.T);
    w.tolv.upload(s.tol_var.data(), s.T);
    w.model_t.upload(s.model_t.data(), s.T);
    w.state.alloc(sizeof(LoopState));
    w.slot.alloc(sizeof(int32_t) * (size_t)(p + hist));
    w.nrow.alloc(sizeof(int32_t) * (size_t)(p + hist));
    const bool head = use_mlp_head(s, d, p);
    int nblk = picard_partial_blocks(d.D, batch);
    if (head && head_slabs(d.D) > nblk) nblk = head_slabs(d.D);
    w.partials.alloc(sizeof(float) * (size_t)nblk * p * batch);
    if (head) {
        w.head_count.alloc(sizeof(int32_t) * (size_t)(head_slabs(d.D) + 1));
        PD_HIP(hipMemset(w.head_count.p, 0, w.head_count.bytes));
    }
    if (s.heun) {
        w.xt.alloc(sizeof(float) * (size_t)p * BD);
        w.eps2.alloc(sizeof(float) * (size_t)p * BD);
        w.model_t_next.upload(s.model_t_next.data(), s.T);
        w.nrow2.alloc(sizeof(int32_t) * (size_t)p);
    }
    if (s.dpm) {
        w.Rt.upload(s.R.data(), s.T);
        w.St.upload(s.S.data(), s.T);
        w.xprev.alloc(sizeof(float) * (size_t)BD);
        w.eprev.alloc(sizeof(float) * (size_t)BD);
    }
    const size_t sc = d.scratch_floats((int64_t)(p + hist) * batch);
    if (sc) w.scratch.alloc(sc * sizeof(float));
    host_mapped(&w.h_state, &w.h_state_dev, 1);
    PD_HIP(hipEventCreateWithFlags(&w.batch_event, hipEventDisableTiming));
    host_mapped(&w.h_trace, &w.h_trace_dev, (size_t)s.T);
}

extern "C" pd_status pd_workspace_create(const pd_schedule* s, const pd_denoiser* d, int32_t p,
                                         int32_t batch, pd_workspace** out) {
    return guard([&] {
        require(s && d && out, "NULL argument");
        *out = nullptr;
        require(p >= 1, "p must be >= 1");
        require(batch >= 1, "batch must be >= 1");
        const int pc = p < s->T ? p : s->T;
        auto w = std::make_unique<pd_workspace>();
        create_workspace(*s, *d, pc, batch, *w);
        *out = w.release();
    });
}

extern "C" void pd_workspace_destroy(pd_workspace* w) { delete w; }

// ============================================================== samplers
static void check_sample_args(const pd_schedule* s, const pd_denoiser* d, int32_t batch,
                              const int64_t* shape, int32_t ndim, const float* x_out) {
    require(s && d, "schedule and denoiser must not be NULL");
    require(batch >= 1, "batch must be >= 1");
    require(shape != nullptr && ndim == (int32_t)d->shape.size(),
            "sample_shape does not match the denoiser");
    for (int i = 0; i < ndim; ++i)
        require(shape[i] == d->shape[i], "sample_shape does not match the denoiser");
    require(s->T_train == d->T_train, "schedule and denoiser disagree on T_train");
    require(x_out != nullptr, "x_out must not be NULL");
}

// Waits for the sampling stream when a sampler leaves, also by an error:
// declared after the workspace it uses, it runs before a workspace made for
// the call is freed, so no queued kernel or copy outlives its buffers.
struct StreamDrain {
    hipStream_t s;
    ~StreamDrain() { (void)hipStreamSynchronize(s); }
};

static pd_workspace* use_workspace(pd_workspace* ws, std::unique_ptr<pd_workspace>& own,
                                   const pd_schedule* s, const pd_denoiser* d, int p, int batch) {
    if (ws) {
        require(ws->s == s && ws->d == d && ws->batch == batch,
                "workspace was made for another schedule, denoiser or batch");
        require(ws->p >= p, "workspace window is smaller than p");
        int dev = 0;
        PD_HIP(hipGetDevice(&dev));
        require(dev == ws->device, "workspace lives on another device");
        return ws;
    }
    own = std::make_unique<pd_workspace>();
    create_workspace(*s, *d, p, batch, *own);
    return own.get();
}

// x_0 into ring slot 0 and every step's noise, in one launch that also starts
// the Picard loop when init is given
static void draw_noise(pd_workspace& w, uint64_t seed, const PicardInit* init, hipStream_t st) {
    const int64_t BD = (int64_t)w.batch * w.D;
    launch_sample_setup(seed, BD, w.ring.as<float>(), (int64_t)w.T * BD, w.zstd.as<float>(), BD,
                        w.noise.as<float>(), init, st);
}

static void fill_stats(pd_sample_stats* stats, int iters, int64_t evals, int batch, bool guided,
                       const int32_t* trace, const KernelTimer& tm) {
    if (!stats) return;
    stats->denoiser_launches = tm.count[CAT_DENOISER];
    stats->update_launches = tm.count[CAT_UPDATE];
    stats->finalize_launches = tm.count[CAT_FINALIZE];
    stats->denoiser_ms = tm.ms[CAT_DENOISER];
    stats->update_ms = tm.ms[CAT_UPDATE];
    stats->finalize_ms = tm.ms[CAT_FINALIZE];
    stats->iters = iters;
    stats->evals_per_sample = evals;
    stats->network_rows = evals * batch * (guided ? 2 : 1);
    if (stats->stride_trace && stats->trace_cap > 0 && trace) {   // host memory, loop finished
        const int n = iters < stats->trace_cap ? iters : stats->trace_cap;
        if (n > 0) std::memcpy(stats->stride_trace, trace, sizeof(int32_t) * n);
    }
}

// The mixture model's whole sampling loop fits in one workgroup's LDS.
static constexpr size_t kFusedLoopLds = 64 * 1024;

static bool use_fused_gmm_loop(const pd_schedule& s, const pd_denoiser& d, int T, int p,
                               int batch) {
    return d.desc.kind == PD_MODEL_GMM2D && !s.heun && !s.dpm &&
           gmm_loop_lds_bytes(T, d.desc.n_components, p, batch) <= kFusedLoopLds;
}

// The stride test's threshold factor c (threshold c sigma^2) and the divisor
// of the summed squared differences (the error is sum / div): the relaxed
// rule of Sec. 3.1 compares the per-dimension mean with tau^2 sigma^2,
// Prop. 2 the squared norm with 4 eps^2 sigma^2 / T^2 (eps = tau).
struct StopTest {
    float factor, err_div;
};
static StopTest stop_test(const pd_schedule& s, float tau, int64_t D) {
    if (s.desc.stop_rule == PD_STOP_PROP2) {
        const double e = (double)tau, T = (double)s.T;
        return StopTest{(float)(4.0 * e * e / (T * T)), 1.0f};
    }
    return StopTest{tau * tau, (float)D};
}

static GmmLoopArgs gmm_loop_args(const pd_schedule& s, const pd_denoiser& d, pd_workspace& w, int p,
                                 int batch, StopTest stop, float* x_out) {
    GmmLoopArgs a;
    a.g = d.gmm();
    a.A = w.A.as<float>();
    a.B = w.B.as<float>();
    a.tol_var = w.tolv.as<float>();
    a.model_t = w.model_t.as<int32_t>();
    a.noise = w.noise.p ? w.noise.as<float>() : nullptr;
    a.x0 = w.ring.as<float>();
    a.out = x_out;
    a.st = w.state.as<LoopState>();
    a.st_host = w.h_state_dev;
    a.trace = w.h_trace_dev;
    a.T = s.T;
    a.p = p;
    a.batch = batch;
    a.tol_offset = s.desc.tol_index_offset;
    a.tau2 = stop.factor;
    a.err_div = stop.err_div;
    return a;
}

extern "C" pd_status pd_sample_sequential(const pd_schedule* s, const pd_denoiser* d,
                                          uint64_t noise_seed, int32_t batch,
                                          const int64_t* sample_shape, int32_t ndim, float* x_out,
                                          pd_sample_stats* stats, pd_workspace* ws, void* stream) {
    return guard([&] {
        check_sample_args(s, d, batch, sample_shape, ndim, x_out);
        if (stats) require(stats->trace_cap >= 0, "trace_cap must be >= 0");
        const hipStream_t st = static_cast<hipStream_t>(stream);
        std::unique_ptr<pd_workspace> own;
        pd_workspace& w = *use_workspace(ws, own, s, d, 1, batch);
        const StreamDrain drain{st};
        const int64_t BD = (int64_t)batch * d->D;
        float* x = w.ring.as<float>();
        KernelTimer tm;
        tm.on = stats && stats->time_kernels;
        tm.st = st;
        draw_noise(w, noise_seed, nullptr, st);
        if (use_fused_gmm_loop(*s, *d, s->T, 1, batch)) {
            tm.mark(-1);
            launch_gmm_sequential_loop(gmm_loop_args(*s, *d, w, 1, batch, StopTest{0.f, 2.f}, x_out), st);
            tm.mark(CAT_UPDATE);
            PD_HIP(hipStreamSynchronize(st));
            tm.collect();
            fill_stats(stats, s->T, s->T, batch, d->guided(), nullptr, tm);
            const int n = stats ? (s->T < stats->trace_cap ? s->T : stats->trace_cap) : 0;
            for (int i = 0; i < n && stats->stride_trace; ++i) stats->stride_trace[i] = 1;
            return;
        }
        tm.mark(-1);
        int64_t evals = 0;
        for (int i = 0; i < s->T; ++i) {
            const RowSrc src{x, nullptr, BD, batch, 1, w.model_t.as<int32_t>() + i, nullptr, d->T_train - 1};
            d->forward(src, w.eps.as<float>(), w.scratch.as<float>(), st);
            ++evals;
            if (s->heun && i + 1 < s->T) {     // Heun: second evaluation at the Euler prediction
                launch_seq_heun_predict(x, w.eps.as<float>(), s->A[i], s->B[i], BD, w.xt.as<float>(), st);
                const RowSrc src2{w.xt.as<float>(), nullptr, BD, batch, 1,
                                  w.model_t_next.as<int32_t>() + i, nullptr, d->T_train - 1};
                d->forward(src2, w.eps2.as<float>(), w.scratch.as<float>(), st);
                launch_seq_heun_combine(w.eps.as<float>(), w.eps2.as<float>(), BD, st);
                ++evals;
            }
            tm.mark(CAT_DENOISER);
            if (s->dpm) {
                launch_seq_step_dpm(x, w.eps.as<float>(), w.xprev.as<float>(), w.eprev.as<float>(),
                                    s->A[i], s->B[i], s->R[i], s->S[i], s->R[i] != 0.f, BD, st);
            } else {
                const float* z = w.noise.p ? w.noise.as<float>() + (int64_t)i * BD : nullptr;
                launch_seq_step(x, w.eps.as<float>(), z, s->A[i], s->B[i], BD, st);
            }
            tm.mark(CAT_UPDATE);
        }
        PD_HIP(hipMemcpyAsync(x_out, x, sizeof(float) * BD, hipMemcpyDeviceToDevice, st));
        PD_HIP(hipStreamSynchronize(st));
        tm.collect();
        if (stats) {
            fill_stats(stats, s->T, evals, batch, d->guided(), nullptr, tm);
            const int n = s->T < stats->trace_cap ? s->T : stats->trace_cap;
            for (int i = 0; i < n && stats->stride_trace; ++i) stats->stride_trace[i] = 1;
        }
    });
}

extern "C" pd_status pd_sample_picard(const pd_schedule* s, const pd_denoiser* d, int32_t p,
                                      float tau, uint64_t noise_seed, int32_t batch,
                                      const int64_t* sample_shape, int32_t ndim, float* x_out,
                                      pd_sample_stats* stats, pd_workspace* ws, void* stream) {
    return guard([&] {
        require(p >= 1, "p must be >= 1");
        require(!std::isnan(tau) && tau >= 0.f, "tau must be >= 0 (inf allowed)");
        check_sample_args(s, d, batch, sample_shape, ndim, x_out);
        if (stats) require(stats->trace_cap >= 0, "trace_cap must be >= 0");
        const int T = s->T;
        const int pc = p < T ? p : T;
        if (pc > 128) fail(PD_ERR_UNSUPPORTED, "windows larger than 128 points are not built");
        const hipStream_t st = static_cast<hipStream_t>(stream);
        std::unique_ptr<pd_workspace> own;
        pd_workspace& w = *use_workspace(ws, own, s, d, pc, batch);
        const StreamDrain drain{st};
        const int64_t BD = (int64_t)batch * d->D;
        const StopTest stop = stop_test(*s, tau, d->D);
        LoopState* dst = w.state.as<LoopState>();

        KernelTimer tm;
        tm.on = stats && stats->time_kernels;
        tm.st = st;
        const bool fused_gmm = use_fused_gmm_loop(*s, *d, T, pc, batch);
        const int32_t* mtn = s->heun ? w.model_t_next.as<int32_t>() : nullptr;
        int32_t* nrow2 = s->heun ? w.nrow2.as<int32_t>() : nullptr;
        const PicardInit init{dst, w.slot.as<int32_t>(), w.nrow.as<int32_t>(), w.model_t.as<int32_t>(),
                              mtn, nrow2, T, pc};
        // the mixture's loop draws x_0 and the noise itself when all of it fits in its LDS
        const bool draw_in_loop =
            fused_gmm && gmm_loop_stages_noise(T, d->desc.n_components, pc, batch, kFusedLoopLds);
        if (!draw_in_loop) draw_noise(w, noise_seed, fused_gmm ? nullptr : &init, st);
        if (fused_gmm) {
            tm.mark(-1);
            const GmmDraw draw{draw_in_loop ? 1 : 0, noise_seed,
                               w.noise.p ? w.zstd.as<float>() : nullptr};
            launch_gmm_picard_loop(gmm_loop_args(*s, *d, w, pc, batch, stop, x_out), draw,
                                   kFusedLoopLds, st);
            tm.mark(CAT_UPDATE);
            PD_HIP(hipStreamSynchronize(st));     // the kernel wrote the state's host copy
            if (w.h_state->status != PD_OK) fail(PD_ERR_NUMERIC, "non-finite point or error in the window");
            tm.collect();
            fill_stats(stats, w.h_state->k, w.h_state->evals, batch, d->guided(), w.h_trace, tm);
            return;
        }
        const RowSrc src2{w.xt.as<float>(), nullptr, BD, batch, pc, nrow2, &dst->p_eff, d->T_train - 1};
        const int hist = s->dpm ? 1 : 0;     // the multistep drift's row x_{t-1}
        const int slots = pc + 1 + hist;
        const float* xT = w.ring.as<float>() + (int64_t)(T % slots) * BD;
        const FinalizeArgs fin{dst, w.h_state_dev, w.partials.as<float>(), pc, batch, d->D, T,
                               w.tolv.as<float>(), stop.factor, stop.err_div, s->desc.tol_index_offset,
                               w.model_t.as<int32_t>(), w.h_trace_dev, w.slot.as<int32_t>(),
                               w.nrow.as<int32_t>(), mtn, nrow2, slots, hist, xT, x_out, BD};
        const bool head = use_mlp_head(*s, *d, pc);
        const RowSrc src{w.ring.as<float>(), w.slot.as<int32_t>(), BD,     batch,
                         pc + hist,          w.nrow.as<int32_t>(), &dst->nrows, d->T_train - 1};
        // The kernels write the loop state into host memory as they go, so
        // the host decides each next batch while the GPU still runs the
        // previous batch's last iteration (it waits on an event recorded
        // before that iteration): the GPU never waits idle for the host.
        volatile LoopState* hs = w.h_state;
        hs->t = 0;              // the copy still holds the previous call's end
        hs->k = 0;
        hs->status = PD_OK;
        hs->first_stride = 0;
        int t_host = 0, k_host = 0, issued = 0;
        for (;;) {
            // every iteration advances t by at most pc, so at least this many
            // more are needed.  Beyond that, enqueue as many as the mean stride
            // after the first predicts (the first window holds copies of x_0 and
            // in practice slides by one), but at most as many as are already
            // done: strides grow as the trajectory converges, so early means
            // overestimate what is left, and iterations enqueued past the end
            // (they find p_eff = 0 on the device and return at once) still cost
            // a dispatch each.  Iterations still queued count against it.
            // The first batch adds one iteration more than the first window's
            // slide of one requires: the host then decides the second batch
            // from two finished iterations (the mean stride) while a third
            // still runs, instead of draining the stream and leaving the GPU
            // idle; it is wasted only when the loop ends within two iterations.
            const int in_flight = issued - k_host;
            int need = (T - t_host + pc - 1) / pc;
            if (issued == 0 && T > 1) need = 2 + (T - 1 + pc - 1) / pc;
            const int first_stride = hs->first_stride;
            if (k_host >= 2 && t_host > first_stride) {
                const double mean = (double)(t_host - first_stride) / (double)(k_host - 1);
                int est = (int)std::ceil((double)(T - t_host) / mean);
                est = est < issued ? est : issued;
                need = need > est ? need : est;
            }
            need = need < T - t_host ? need : T - t_host;   // stride >= 1 bounds the rest
            need -= in_flight;
            if (issued + need > T) need = T - issued;
            if (need > 0) {
                tm.mark(-1);
                for (int it = 0; it < need; ++it) {
                    if (it == need - 1) PD_HIP(hipEventRecord(w.batch_event, st));
                    if (head) {
                        // the last layer with the update, error, stride and slide
                        const float* h = d->mlp_trunk(src, w.scratch.as<float>(), st);
                        tm.mark(CAT_DENOISER);
                        const HeadScanArgs ha{d->mlp_head(), h, src, dst, w.ring.as<float>(),
                                              w.eps.as<float>(), w.noise.as<float>(), w.A.as<float>(),
                                              w.B.as<float>(), batch, d->D, w.partials.as<float>(),
                                              w.head_count.as<int32_t>(), head_slabs(d->D)};
                        launch_mlp_head_scan(ha, fin, st);
                        tm.mark(CAT_UPDATE);
                        continue;
                    }
                    if (s->heun && d->desc.kind == PD_MODEL_MLP) {
                        // the MLP's last layer also writes every row's Euler prediction
                        const HeunPredictArgs hp{dst, w.ring.as<float>(), w.A.as<float>(),
                                                 w.B.as<float>(), slots, w.xt.as<float>()};
                        launch_linear_dense_predict(d->mlp_head(),
                                                    d->mlp_trunk(src, w.scratch.as<float>(), st),
                                                    src, hp, w.eps.as<float>(), st);
                    } else {
                        d->forward(src, w.eps.as<float>(), w.scratch.as<float>(), st);
                        if (s->heun)
                            launch_heun_predict(dst, w.ring.as<float>(), w.eps.as<float>(),
                                                w.A.as<float>(), w.B.as<float>(), pc, BD,
                                                w.xt.as<float>(), st);
                    }
                    // Heun: the second evaluation, at every row's Euler prediction
                    if (s->heun) d->forward(src2, w.eps2.as<float>(), w.scratch.as<float>(), st);
                    tm.mark(CAT_DENOISER);
                    const bool fused = launch_picard_scan(
                        dst, w.ring.as<float>(), w.eps.as<float>(), w.noise.as<float>(),
                        w.A.as<float>(), w.B.as<float>(), w.Rt.as<float>(), w.St.as<float>(), pc,
                        batch, d->D, w.partials.as<float>(), fin,
                        s->heun ? w.eps2.as<float>() : nullptr, st);   // Heun: the scan averages
                    tm.mark(CAT_UPDATE);
                    if (!fused) {
                        launch_picard_finalize(fin, st);
                        tm.mark(CAT_FINALIZE);
                    }
                }
                issued += need;
                // every iteration but the batch's last has run: decide the
                // next batch while that one runs
                PD_HIP(hipEventSynchronize(w.batch_event));
            } else if (in_flight > 0) {
                PD_HIP(hipStreamSynchronize(st));   // the queued ones may finish the loop
            } else {
                fail(PD_ERR_DEVICE, "Picard loop did not terminate within T iterations");
            }
            k_host = hs->k;
            t_host = hs->t;
            if (t_host >= T || hs->status != PD_OK) break;
        }
        PD_HIP(hipStreamSynchronize(st));     // every queued launch (the last wrote x_T out)
        if (w.h_state->status != PD_OK) fail(PD_ERR_NUMERIC, "non-finite point or error in the window");
        if (w.h_state->t < T) fail(PD_ERR_DEVICE, "Picard loop did not reach T");
        const int iters = w.h_state->k;
        const int64_t evals = w.h_state->evals;
        tm.collect();
        fill_stats(stats, iters, evals, batch, d->guided(), w.h_trace, tm);
    });
}
