"""Pins for the oracle's DDPM / DDIM tables.

Each check is a property the tables must satisfy (marginal consistency of the
forward process, a known identity between the two samplers, exact recovery of
a point mass), not a restatement of the formulas used to build them.
"""
import math

import numpy as np
import pytest

from oracle import denoisers, samplers, schedule


def _next_abar(tb, i):
    """abar at the network timestep the chain reaches after reverse step i."""
    return tb.alphabar[tb.model_t[i + 1]] if i + 1 < tb.T else 1.0


def test_beta_endpoints_and_product():
    b = schedule.betas(1000, 1e-4, 0.02)
    assert b[0] == 1e-4 and abs(b[-1] - 0.02) < 1e-17
    assert np.allclose(np.diff(b), (0.02 - 1e-4) / 999, rtol=0, atol=1e-17)
    ab = schedule.alphabars(b)
    assert np.allclose(ab, np.exp(np.cumsum(np.log1p(-b))), rtol=1e-12, atol=0)
    assert abs(ab[-1] - 4.036e-5) < 1e-8           # value quoted for T=1000


@pytest.mark.parametrize("tb", [schedule.ddpm(100), schedule.ddpm(1000),
                                schedule.ddim(1000, 200, 0.0), schedule.ddim(1000, 200, 1.0),
                                schedule.ddim(1000, 50, 0.5)],
                         ids=["ddpm100", "ddpm1000", "ddim200e0", "ddim200e1", "ddim50e05"])
def test_marginal_consistency(tb):
    """With point-mass data mu and its exact eps, a step maps the forward
    marginal N(sqrt(ab_n) mu, (1-ab_n) I) onto the marginal at the next
    timestep: mean and variance of the affine update must match."""
    for i in range(tb.T):
        an = tb.alphabar[tb.model_t[i]]
        anext = _next_abar(tb, i)
        # x' = (1 + A) x + B eps,  eps = (x - sqrt(an) mu) / sqrt(1 - an)
        g = 1.0 + tb.A[i] + tb.B[i] / math.sqrt(1.0 - an)
        h = -tb.B[i] * math.sqrt(an) / math.sqrt(1.0 - an)
        assert abs(g * math.sqrt(an) + h - math.sqrt(anext)) < 1e-12, i
        assert abs(g * g * (1.0 - an) + tb.noise_var[i] - (1.0 - anext)) < 1e-12, i


def test_model_timesteps():
    assert np.array_equal(schedule.ddpm(10).model_t, np.arange(9, -1, -1))
    d = schedule.ddim(1000, 200)
    assert d.model_t[0] == 995 and d.model_t[-1] == 0
    assert np.all(np.diff(d.model_t) == -5)


def test_ddim_eta1_full_chain_is_ddpm():
    """Song et al.: DDIM with eta = 1 on the full chain is DDPM's ancestral sampler."""
    a, b = schedule.ddpm(1000), schedule.ddim(1000, 1000, 1.0)
    for f in ("A", "B", "noise_var", "tol_var"):
        assert np.allclose(getattr(a, f), getattr(b, f), rtol=1e-10, atol=1e-14), f
    assert np.array_equal(a.model_t, b.model_t)


def test_variances():
    d = schedule.ddpm(1000)
    assert d.noise_var[-1] == 0.0 and np.all(d.noise_var[:-1] > 0)
    s = np.sqrt(d.noise_var)
    assert abs(s[0] - 0.1414) < 1e-3 and abs(s[-2] - 7.38e-3) < 1e-5
    e = schedule.ddim(1000, 200, 0.0)
    assert np.all(e.noise_var == 0.0)
    assert e.tol_var[-1] == 0.0 and np.all(e.tol_var[:-1] > 0)
    assert abs(e.tol_var[0] - 0.0955) < 5e-4


def test_ddim_rejects_non_divisor():
    with pytest.raises(ValueError):
        schedule.ddim(1000, 300)


@pytest.mark.parametrize("tb", [schedule.ddpm(50), schedule.ddim(500, 50, 0.0)],
                         ids=["ddpm", "ddim"])
def test_point_mass_recovered_exactly(tb):
    """Data = delta at mu: both update forms, driven by the exact eps, end on mu."""
    mu = np.array([[1.5, -0.25]])
    eps = lambda x, n: denoisers.gmm2d_eps(x, n, tb.alphabar, mu, 0.0, np.float64)
    rng = np.random.default_rng(0)
    x0 = rng.standard_normal((3, 2))
    z = np.sqrt(tb.noise_var)[:, None, None] * rng.standard_normal((tb.T, 3, 2))
    out = samplers.sequential(tb, eps, x0, z, np.float64)
    assert np.allclose(out, mu, atol=1e-9)
    out2 = samplers.sequential_mean_form(tb, eps, x0, z)
    assert np.allclose(out2, out, atol=1e-10)


def test_drift_form_matches_textbook_means():
    tb = schedule.ddpm(200)
    means = np.array([[2.0, 0.0], [-1.0, 1.0]])
    eps = lambda x, n: denoisers.gmm2d_eps(x, n, tb.alphabar, means, 0.5, np.float64)
    rng = np.random.default_rng(1)
    x0 = rng.standard_normal((4, 2))
    z = np.sqrt(tb.noise_var)[:, None, None] * rng.standard_normal((tb.T, 4, 2))
    a = samplers.sequential(tb, eps, x0, z, np.float64)
    b = samplers.sequential_mean_form(tb, eps, x0, z)
    assert np.allclose(a, b, rtol=1e-11, atol=1e-11)
