"""Pins of the oracle's Heun drift (Sec. 3.3: the Euler step of Algorithm 1's
drift swapped for Heun's method, here on the DDIM probability-flow ODE).

For Gaussian data N(mu, s^2 I) the ODE has a closed form: in the coordinates
xbar = x / sqrt(abar), sig = sqrt(1 - abar) / sqrt(abar) the flow maps
xbar - mu -> (xbar - mu) sqrt(s^2 + sig^2) / sqrt(s^2 + sig0^2).  Heun's step
is second order and the DDIM (Euler) step first order, so halving the step
size must divide their errors by about 4 and 2; the single Euler final step
adds a local error of the same second order."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import Problem, samplers, schedule


def _gauss(T, solver, dtype=np.float64, batch=3, seed=0, T_train=1200):
    sch = W.ScheduleSpec("ddim", T_train, T, solver=solver)
    m = W.ModelSpec("gmm2d", (2,), n_components=1, radius=1.5, sigma0=0.7)
    wl = W.Workload("gauss", sch, m, p=8, tau=0.1, batch=batch, noise_seed=seed)
    return Problem(wl, W.make_weights(m), dtype)


def _exact(pr):
    means, s = W.gmm_components(pr.w.model)
    ab0 = pr.tables.alphabar[pr.tables.model_t[0]]
    sig0sq = (1.0 - ab0) / ab0
    xbar0 = pr.x0.astype(np.float64) / math.sqrt(ab0)
    return means[0] + (xbar0 - means[0]) * (s / math.sqrt(s * s + sig0sq))


def _errors(solver, Ts):
    out = []
    for T in Ts:
        pr = _gauss(T, solver)
        out.append(float(np.max(np.abs(pr.sequential() - _exact(pr)))))
    return out


def test_heun_is_second_order_and_ddim_first_order():
    Ts = [10, 20, 40, 80]
    eh = _errors("heun", Ts)
    ee = _errors("euler", Ts)
    rh = [eh[i] / eh[i + 1] for i in range(3)]
    re = [ee[i] / ee[i + 1] for i in range(3)]
    assert all(3.0 < r < 5.5 for r in rh[1:]), rh
    assert all(1.6 < r < 2.6 for r in re[1:]), re
    assert eh[-1] < 0.1 * ee[-1]


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_heun_window_of_one_is_sequential_bitwise(dtype):
    pr = _gauss(30, "heun", dtype=dtype)
    r = pr.picard(p=1, tau=0.1)
    assert r.iters == 30 and r.trace == [1] * 30
    assert np.array_equal(r.x, pr.sequential())
    assert r.evals == 2 * 30 - 1                  # two per step, one for the last


def test_heun_zero_tolerance_reproduces_sequential():
    pr = _gauss(24, "heun")
    r = pr.picard(p=24, tau=0.0)
    assert r.iters <= 24
    assert np.allclose(r.x, pr.sequential(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("p", [3, 7, 40])
def test_heun_evaluation_count(p):
    pr = _gauss(40, "heun", dtype=np.float32)
    r = pr.picard(p=p)
    t, ev = 0, 0
    for s in r.trace:
        pe = min(p, 40 - t)
        ev += 2 * pe - (1 if t + pe == 40 else 0)
        t += s
    assert t == 40 and r.evals == ev


def test_heun_drift_definition():
    """One step written out: Euler prediction, then the averaged epsilon;
    the last step keeps the Euler drift."""
    pr = _gauss(12, "heun")
    tb = pr.tables
    A, Bc = tb.A, tb.B
    x = pr.x0
    for i in (0, 5, 11):
        y, nev, _ = samplers.drifts(tb, A, Bc, pr.eps, x[None], np.array([i]))
        e = pr.eps(x, np.full(x.shape[0], tb.model_t[i]))
        if i < 11:
            xt = x + (A[i] * x + Bc[i] * e)
            e2 = pr.eps(xt, np.full(x.shape[0], tb.model_t[i + 1]))
            ref = A[i] * x + (0.5 * Bc[i]) * (e + e2)
            assert nev == 2
        else:
            ref = A[i] * x + Bc[i] * e
            assert nev == 1
        assert np.array_equal(y[0], ref)


def test_heun_needs_the_ode():
    with pytest.raises(ValueError):
        schedule.ddim(100, 10, eta=0.5, solver="heun")
    assert schedule.ddim(100, 10, solver="heun").model_t_next[-1] == -1
