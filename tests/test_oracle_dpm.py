"""Pins of the oracle's DPM-Solver++(2M) drift (the paper's ParaDPMSolver:
DPMSolver steps solved by Picard iteration, Sec. 4), on the eta = 0 DDIM
chain.  The closed-form flow of Gaussian data (see test_oracle_heun.py) fixes
the order: second order, so halving the step divides the error by about 4."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import Problem, schedule
from test_oracle_heun import _exact


def _gauss(T, solver, dtype=np.float64, batch=3, seed=0, T_train=1200):
    sch = W.ScheduleSpec("ddim", T_train, T, solver=solver)
    m = W.ModelSpec("gmm2d", (2,), n_components=1, radius=1.5, sigma0=0.7)
    wl = W.Workload("gauss", sch, m, p=8, tau=0.1, batch=batch, noise_seed=seed)
    return Problem(wl, W.make_weights(m), dtype)


def test_dpm_solver_is_second_order():
    errs = []
    for T in (20, 40, 80, 160):
        pr = _gauss(T, "dpm2m", T_train=1600)
        errs.append(float(np.max(np.abs(pr.sequential() - _exact(pr)))))
    ratios = [errs[i] / errs[i + 1] for i in range(3)]
    assert all(3.0 < r < 5.5 for r in ratios[1:]), (errs, ratios)
    ddim = _gauss(160, "euler", T_train=1600)
    assert errs[-1] < 0.5 * float(np.max(np.abs(ddim.sequential() - _exact(ddim))))


def test_drift_table_equals_data_prediction_form():
    """The P, Q, R, S tables against the solver written in its own terms:
    x0 = (x - sig eps)/alpha, D = (1 + 1/2r) x0_i - (1/2r) x0_{i-1},
    x_{i+1} = (sig_{i+1}/sig_i) x_i - alpha_{i+1} (exp(-h) - 1) D, first
    order at the first step, x0 itself at the last."""
    T = 12
    pr = _gauss(T, "dpm2m")
    tb = pr.tables
    ab, c = tb.alphabar, tb.T_train // T
    x = pr.x0.astype(np.float64)
    x0_prev = lam_prev = None
    for i in range(T):
        n = int(tb.model_t[i])
        a, sg = math.sqrt(ab[n]), math.sqrt(1.0 - ab[n])
        lam = math.log(a / sg)
        x0 = (x - sg * pr.eps(x, np.full(x.shape[0], n))) / a
        if n - c < 0:
            x = x0
        else:
            a1, s1 = math.sqrt(ab[n - c]), math.sqrt(1.0 - ab[n - c])
            h = math.log(a1 / s1) - lam
            if i == 0:
                D = x0
            else:
                r = (lam - lam_prev) / h
                D = (1.0 + 1.0 / (2.0 * r)) * x0 - (1.0 / (2.0 * r)) * x0_prev
            x = (s1 / sg) * x - a1 * math.expm1(-h) * D
        x0_prev, lam_prev = x0, lam
    assert np.allclose(pr.sequential(), x, rtol=1e-12, atol=1e-12)


def test_first_and_last_steps_are_ddim():
    d = schedule.ddim(1000, 40, solver="dpm2m")
    e = schedule.ddim(1000, 40)
    for i in (0, 39):
        assert d.A[i] == e.A[i] and d.B[i] == e.B[i] and d.R[i] == 0 and d.S[i] == 0
    assert np.all(d.R[1:39] != 0)
    # the data-prediction form: R x + S eps of the previous step is a multiple of x0_{i-1}
    ab = d.alphabar
    for i in (1, 17, 38):
        n_prev = int(d.model_t[i - 1])
        assert math.isclose(d.S[i] / d.R[i], -math.sqrt(1.0 - ab[n_prev]), rel_tol=1e-12)


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_dpm_window_of_one_is_sequential_bitwise(dtype):
    pr = _gauss(30, "dpm2m", dtype=dtype)
    r = pr.picard(p=1, tau=0.1)
    assert r.iters == 30 and r.trace == [1] * 30
    assert np.array_equal(r.x, pr.sequential())
    assert r.evals == 30 + 29          # every iteration after the first re-evaluates x_{t-1}


def test_dpm_zero_tolerance_reproduces_sequential():
    pr = _gauss(24, "dpm2m")
    r = pr.picard(p=24, tau=0.0)
    assert r.iters <= 24
    assert np.allclose(r.x, pr.sequential(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("p", [3, 7, 40])
def test_dpm_evaluation_count(p):
    pr = _gauss(40, "dpm2m", dtype=np.float32)
    r = pr.picard(p=p)
    t, ev = 0, 0
    for s in r.trace:
        ev += min(p, 40 - t) + (1 if t >= 1 else 0)
        t += s
    assert t == 40 and r.evals == ev


def test_dpm_needs_the_ode():
    with pytest.raises(ValueError):
        schedule.ddim(100, 10, eta=0.3, solver="dpm2m")
