"""Pins for the oracle's sequential chain and its Algorithm 1 Picard solver."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import Problem, denoisers, philox, samplers, schedule

INF = float("inf")


# ---------------------------------------------------------------- stride rule
def _err(*rows):
    rows = [[r] if np.isscalar(r) else list(r) for r in rows]
    return np.array([[0.0] * len(rows[0])] + rows, dtype=np.float64)


@pytest.mark.parametrize("err,tol,expect", [
    (_err(0.1, 0.1, 0.1), [0, 1, 1, 1], 4),          # all pass -> p_eff
    (_err(2.0, 0.1, 0.1), [0, 1, 1, 1], 1),          # first tested offset fails
    (_err(0.1, 0.1, 5.0), [0, 1, 1, 1], 3),          # later offset fails
    (_err(1.0, 1.0, 1.0), [0, 1, 1, 1], 4),          # equality passes
    (_err(0.1, np.nan, 0.1), [0, 1, 1, 1], 2),       # NaN fails
    (_err([0.1, 3.0], [0.1, 0.1]), [0, 1, 1], 1),    # any sample of the batch fails
    (_err([0.1, 0.2], [0.1, 0.2]), [0, 1, 1], 3),
])
def test_stride_rule_table(err, tol, expect):
    assert samplers.stride_from_errors(err, np.array(tol, float), err.shape[0]) == expect


def test_stride_rule_window_of_one():
    assert samplers.stride_from_errors(np.zeros((1, 1)), np.zeros(1), 1) == 1


# ------------------------------------------------------------------- fixtures
def _gmm_problem(T=30, dtype=np.float64, batch=1, kind="ddpm", seed=0):
    sch = W.ScheduleSpec(kind, T if kind == "ddpm" else 5 * T, T)
    wl = W.Workload("t", sch, W.ModelSpec("gmm2d", (2,)), p=8, tau=0.1,
                    batch=batch, noise_seed=seed)
    return Problem(wl, W.make_weights(wl.model), dtype)


def _mlp_problem(T=25, dtype=np.float32, batch=2):
    wl = W.Workload("t", W.ScheduleSpec("ddpm", T, T),
                    W.ModelSpec("mlp", (4, 3), width=32, weight_seed=4),
                    p=6, tau=0.1, batch=batch, noise_seed=3)
    return Problem(wl, W.make_weights(wl.model), dtype)


def _conv_problem(T=20, dtype=np.float32, batch=1, kind="ddpm"):
    sch = W.ScheduleSpec(kind, T if kind == "ddpm" else 5 * T, T)
    wl = W.Workload("t", sch, W.ModelSpec("conv1x1", (4, 5, 6), width=16, weight_seed=2),
                    p=5, tau=0.1, batch=batch, noise_seed=1)
    return Problem(wl, W.make_weights(wl.model), dtype)


PROBLEMS = {"gmm": _gmm_problem, "mlp": _mlp_problem, "conv": _conv_problem}


# --------------------------------------------------------------- equivalences
@pytest.mark.parametrize("name", list(PROBLEMS))
@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_window_of_one_is_sequential_bitwise(name, dtype):
    pr = PROBLEMS[name](dtype=dtype)
    r = pr.picard(p=1, tau=0.1)
    assert r.iters == pr.tables.T and r.trace == [1] * pr.tables.T
    assert np.array_equal(r.x, pr.sequential())


@pytest.mark.parametrize("name", list(PROBLEMS))
def test_zero_tolerance_reproduces_sequential(name):
    pr = PROBLEMS[name](dtype=np.float64)
    T = pr.tables.T
    r = pr.picard(p=T, tau=0.0)
    assert r.iters <= T
    seq = pr.sequential()
    assert np.allclose(r.x, seq, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("name", list(PROBLEMS))
@pytest.mark.parametrize("p", [1, 3, 7, 100])
def test_iteration_count_bounds_and_trace(name, p):
    pr = PROBLEMS[name](dtype=np.float32)
    T = pr.tables.T
    r = pr.picard(p=p)
    assert math.ceil(T / p) <= r.iters <= T
    assert sum(r.trace) == T and all(1 <= s <= p for s in r.trace)
    # evals = sum of window sizes min(p, T - t)
    t, ev = 0, 0
    for s in r.trace:
        ev += min(p, T - t); t += s
    assert r.evals == ev


@pytest.mark.parametrize("name", list(PROBLEMS))
@pytest.mark.parametrize("p", [1, 4, 9])
def test_infinite_tolerance_closed_form(name, p):
    """tau = inf: every iteration slides a full window, so each window is one
    Picard sweep from copies of its left end:
    x_{t+j+1} = x_t + sum_{i=t}^{t+j} (A_i x_t + B_i eps(x_t, n_i)) + sum z_i."""
    pr = PROBLEMS[name](dtype=np.float64)
    tb, T = pr.tables, pr.tables.T
    r = pr.picard(p=p, tau=INF, tol_offset=-1)
    assert r.iters == math.ceil(T / p)
    assert r.trace == [min(p, T - p * k) for k in range(r.iters)]
    # with sigma_{t+j}: the noise-free last step x_{T-1} needs an exact match,
    # so the last window stops one short and a one-point window follows
    r0 = pr.picard(p=p, tau=INF, tol_offset=0)
    m = (T - 1) // p
    rem = T - p * m
    expect = [p] * m + ([rem - 1, 1] if rem >= 2 else [1])
    assert r0.trace == expect
    x = pr.x0.copy()
    B = x.shape[0]
    for t in range(0, T, p):
        acc_y = np.zeros_like(x); acc_z = np.zeros_like(x)
        for i in range(t, min(t + p, T)):
            e = pr.eps(x, np.full(B, tb.model_t[i]))
            acc_y = acc_y + (tb.A[i] * x + tb.B[i] * e)
            acc_z = acc_z + pr.noise[i]
        x = x + acc_y + acc_z
    assert np.allclose(r.x, x, rtol=1e-12, atol=1e-12)


def test_linear_gaussian_error_recursion():
    """Data N(0, I): eps = sqrt(1 - abar) x, so the drift is c_i x with
    c_i = A_i + B_i sqrt(1 - abar_{n_i}).  For every iteration the deviation
    from the sequential chain x* obeys
        x^{k+1}_{t+j+1} - x*_{t+j+1} = (x^k_t - x*_t) + sum_{i=t}^{t+j} c_i (x^k_i - x*_i)."""
    tb = schedule.ddpm(40)
    eps = lambda x, n: denoisers.gmm2d_eps(x, n, tb.alphabar, np.zeros((1, 2)), 1.0)
    c = tb.A + tb.B * np.sqrt(1.0 - tb.alphabar[tb.model_t])
    rng = np.random.default_rng(5)
    x0 = rng.standard_normal((2, 2))
    z = np.sqrt(tb.noise_var)[:, None, None] * rng.standard_normal((40, 2, 2))
    xs = [x0]
    for i in range(40):
        xs.append(xs[-1] + c[i] * xs[-1] + z[i])
    xs = np.array(xs)
    seen = []

    def check(k, t, pe, xo, xn, err, stride):
        e_old = xo - xs[t:t + pe + 1]
        pred = e_old[0] + np.cumsum(c[t:t + pe, None, None] * e_old[:pe], axis=0)
        assert np.allclose(xn - xs[t + 1:t + pe + 1], pred, rtol=0, atol=1e-11)
        seen.append(k)

    r = samplers.picard(tb, eps, x0, z, p=12, tau=0.05, dtype=np.float64, on_iter=check)
    assert len(seen) == r.iters and r.iters > math.ceil(40 / 12)


def test_first_k_points_exact_after_k_iterations():
    """The remark after Prop. 1: after k iterations the leading points equal the
    sequential chain.  With tau = 0 on a full window every accepted point is
    exact, so the window start t always sits on sequential values."""
    pr = _gmm_problem(T=25)
    xs = [pr.x0]
    for i in range(25):
        e = pr.eps(xs[-1], np.full(1, pr.tables.model_t[i]))
        xs.append(xs[-1] + (pr.tables.A[i] * xs[-1] + pr.tables.B[i] * e) + pr.noise[i])

    def check(k, t, pe, xo, xn, err, stride):
        assert t >= k                                   # at least one new exact point per iteration
        assert np.allclose(xo[0], xs[t], atol=1e-13)    # left end is exact
        assert np.allclose(xn[0], xs[t + 1], atol=1e-13)  # first new point is exact (Prop. 1)

    pr.picard(p=25, tau=0.0, on_iter=check)


# ----------------------------------------------------------------- brute force
def _brute_picard(tb, eps_fn, x0, z, p, tau, rule="relaxed"):
    """Algorithm 1 with explicit loops over single points and offsets; with
    rule="prop2" the stride test is Prop. 2's |dx|^2 <= 4 eps^2 sigma^2 / T^2
    (eps = tau)."""
    T = tb.T
    x = {0: x0.copy()}
    for i in range(1, min(p, T) + 1):
        x[i] = x0.copy()
    t, k, trace = 0, 0, []
    while t < T:
        pe = min(p, T - t)
        ys = []
        for j in range(pe):
            e = eps_fn(x[t + j], np.full(x0.shape[0], tb.model_t[t + j]))
            ys.append(tb.A[t + j] * x[t + j] + tb.B[t + j] * e)
        new = {}
        sy = np.zeros_like(x0); sz = np.zeros_like(x0)
        for j in range(pe):
            sy = sy + ys[j]; sz = sz + z[t + j]
            new[t + j + 1] = x[t] + sy + sz
        stride = pe
        for j in range(1, pe):
            d = new[t + j] - x[t + j]
            s2 = tb.tol_var[t + j]
            if rule == "prop2":
                errs = (d * d).sum(axis=1)
                thr = 4 * tau ** 2 * s2 / T ** 2 if s2 > 0 else 0.0
            else:
                errs = (d * d).sum(axis=1) / d.shape[1]
                thr = tau * tau * s2 if s2 > 0 else 0.0
            if any(not (e <= thr) for e in errs):
                stride = j
                break
        x.update(new)
        for j in range(1, stride + 1):
            if t + pe + j <= T:
                x[t + pe + j] = x[t + pe].copy()
        t += stride; k += 1; trace.append(stride)
    return x[T], k, trace


@pytest.mark.parametrize("T", [1, 2, 3, 4])
@pytest.mark.parametrize("tau", [0.0, 0.1, INF])
@pytest.mark.parametrize("kind", ["ddpm", "ddim"])
def test_brute_force_tiny(T, tau, kind):
    pr = _gmm_problem(T=T, batch=2, kind=kind, seed=T)
    for p in range(1, T + 1):
        r = pr.picard(p=p, tau=tau)
        xb, kb, tb_ = _brute_picard(pr.tables, pr.eps, pr.x0, pr.noise, p, tau)
        assert (r.iters, r.trace) == (kb, tb_)
        assert np.allclose(r.x, xb, rtol=1e-13, atol=1e-13)
        assert math.ceil(T / p) <= r.iters <= T


def test_tolerance_offset_reading_avoids_zero_variance():
    pr = _mlp_problem(T=25, dtype=np.float64)
    a = pr.picard(p=25, tau=0.1, tol_offset=0)
    b = pr.picard(p=25, tau=0.1, tol_offset=-1)
    assert a.trace[-1] == 1          # sigma_{T-1} = 0 forces a final one-point window
    assert b.iters <= a.iters


def test_non_finite_is_reported():
    pr = _gmm_problem(T=10)
    bad = lambda x, n: np.where(n[:, None] < 3, np.nan, pr.eps(x, n))
    with pytest.raises(samplers.NumericError):
        samplers.picard(pr.tables, bad, pr.x0, pr.noise, 4, 0.1, np.float64)
    with pytest.raises(samplers.NumericError):
        samplers.sequential(pr.tables, bad, pr.x0, pr.noise, np.float64)


def test_noise_is_scaled_step_normals():
    pr = _gmm_problem(T=10, batch=2)
    n = philox.step_normals(0, 10, 2, 2).astype(np.float64)
    assert np.allclose(pr.noise, np.sqrt(pr.tables.noise_var)[:, None, None] * n, rtol=1e-7)
    assert np.all(pr.noise[-1] == 0.0)


def test_prop1_drift_independent_of_position():
    """Prop. 1: if the drifts at the current guess equal those at the true
    solution, one sweep yields the exact window.  With eps chosen so that
    A_i x + B_i eps = B_i (no x-dependence) every sweep from an exact left end
    is exact, so every tested point that the previous sweep already computed
    has (numerically) zero error and passes: stride >= f_prev - t + 1."""
    tb = schedule.ddpm(30)
    ratio = {int(n): tb.A[i] / tb.B[i] for i, n in enumerate(tb.model_t)}
    eps = lambda x, n: -np.array([ratio[int(v)] for v in n])[:, None] * x + 1.0
    rng = np.random.default_rng(2)
    x0 = rng.standard_normal((1, 3))
    z = np.sqrt(tb.noise_var)[:, None, None] * rng.standard_normal((30, 1, 3))
    xs = [x0]
    for i in range(30):
        xs.append(xs[-1] + tb.B[i] + z[i])
    xs = np.array(xs)
    state = {"f": 0, "n": 0}

    def check(k, t, pe, xo, xn, err, stride):
        assert np.allclose(xo[0], xs[t], atol=1e-12)          # exact left end
        assert np.allclose(xn, xs[t + 1:t + pe + 1], atol=1e-12)
        assert stride >= min(state["f"] - t + 1, pe)
        state["f"] = t + pe
        state["n"] += stride > 1

    r = samplers.picard(tb, eps, x0, z, p=5, tau=0.1, dtype=np.float64,
                        tol_offset=-1, on_iter=check)
    assert state["n"] >= 4 and r.iters < 30
    assert np.allclose(r.x, xs[30], atol=1e-12)


@pytest.mark.parametrize("tau", [0.1, 0.5, 2.0])
@pytest.mark.parametrize("p", [3, 8])
def test_brute_force_longer_chains(tau, p):
    for kind in ("ddpm", "ddim"):
        pr = _gmm_problem(T=24, batch=2, kind=kind, seed=11)
        r = pr.picard(p=p, tau=tau)
        xb, kb, tb_ = _brute_picard(pr.tables, pr.eps, pr.x0, pr.noise, p, tau)
        assert (r.iters, r.trace) == (kb, tb_)
        assert np.allclose(r.x, xb, rtol=1e-13, atol=1e-13)


# ------------------------------------------------- Prop. 2's stopping rule
@pytest.mark.parametrize("T", [1, 2, 3, 4])
@pytest.mark.parametrize("eps", [0.0, 1.0, 30.0, INF])
@pytest.mark.parametrize("kind", ["ddpm", "ddim"])
def test_prop2_brute_force_tiny(T, eps, kind):
    pr = _gmm_problem(T=T, batch=2, kind=kind, seed=T + 7)
    for p in range(1, T + 1):
        r = pr.picard(p=p, tau=eps, rule="prop2")
        xb, kb, tb_ = _brute_picard(pr.tables, pr.eps, pr.x0, pr.noise, p, eps, "prop2")
        assert (r.iters, r.trace) == (kb, tb_)
        assert np.allclose(r.x, xb, rtol=1e-13, atol=1e-13)
        assert math.ceil(T / p) <= r.iters <= T


@pytest.mark.parametrize("eps", [1.0, 5.0, 20.0])
def test_prop2_brute_force_longer_chains(eps):
    for kind in ("ddpm", "ddim"):
        pr = _gmm_problem(T=24, batch=2, kind=kind, seed=13)
        r = pr.picard(p=8, tau=eps, rule="prop2")
        xb, kb, tb_ = _brute_picard(pr.tables, pr.eps, pr.x0, pr.noise, 8, eps, "prop2")
        assert (r.iters, r.trace) == (kb, tb_)
        assert np.allclose(r.x, xb, rtol=1e-13, atol=1e-13)


def _pow2_problem(kind, dtype):
    """D = 16 (sqrt D = 4) and T a power of two, so that tau = 2 eps / (T sqrt D)
    and every threshold are exact binary fractions."""
    sch = W.ScheduleSpec("ddpm", 32, 32) if kind == "ddpm" else W.ScheduleSpec("ddim", 64, 16)
    wl = W.Workload("t", sch, W.ModelSpec("mlp", (4, 4), width=32, weight_seed=9),
                    p=8, tau=0.1, batch=2, noise_seed=4)
    return Problem(wl, W.make_weights(wl.model), dtype)


@pytest.mark.parametrize("kind", ["ddpm", "ddim"])
@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("eps", [0.5, 4.0, 64.0, 1024.0])
def test_prop2_equals_relaxed_rule_at_matching_tau(kind, dtype, eps):
    """Prop. 2 bounds the squared norm |dx|^2 by 4 eps^2 sigma^2 / T^2; the
    relaxed rule bounds (1/D) |dx|^2 by tau^2 sigma^2.  The two tests are the
    same inequality when tau = 2 eps / (T sqrt D): the same strides and the
    same sample, bit for bit (every scaling here is by a power of two)."""
    pr = _pow2_problem(kind, dtype)
    T, D = pr.tables.T, pr.D
    tau = 2.0 * eps / (T * math.sqrt(D))
    a = pr.picard(tau=eps, rule="prop2")
    b = pr.picard(tau=tau, rule="relaxed")
    assert (a.iters, a.trace, a.evals) == (b.iters, b.trace, b.evals)
    assert np.array_equal(a.x, b.x)
    # the sqrt(D) factor matters: the relaxed rule at tau = 2 eps / T (no
    # sqrt D) is a looser test and slides further on these inputs
    c = pr.picard(tau=2.0 * eps / T, rule="relaxed")
    assert c.iters <= a.iters


@pytest.mark.parametrize("name", list(PROBLEMS))
def test_prop2_infinite_bound_is_infinite_tolerance(name):
    """eps = inf accepts every point whose sigma^2 > 0, as tau = inf does."""
    pr = PROBLEMS[name](dtype=np.float64)
    a = pr.picard(p=4, tau=INF, rule="prop2")
    b = pr.picard(p=4, tau=INF)
    assert a.trace == b.trace and np.array_equal(a.x, b.x)


def test_prop2_zero_bound_reproduces_sequential():
    pr = _mlp_problem(T=20, dtype=np.float64, batch=1)
    r = pr.picard(p=20, tau=0.0, rule="prop2")
    assert r.iters <= 20
    assert np.allclose(r.x, pr.sequential(), rtol=1e-12, atol=1e-12)


def test_overflowing_error_is_reported():
    """Huge but finite points whose squared differences overflow float32: the
    error is non-finite, and the run stops with NumericError."""
    pr = _conv_problem(T=10, dtype=np.float32)
    w = dict(pr.weights)
    w["b4"] = np.full_like(w["b4"], 1e20)
    wl = pr.w
    pr2 = Problem(wl, w, np.float32)
    with pytest.raises(samplers.NumericError, match="error"):
        pr2.picard()
