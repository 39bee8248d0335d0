"""Pins for the oracle's synthetic denoisers."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import logsumexp

import workloads as W
from oracle import denoisers, schedule


def _log_q(x, n, ab, means, s0):
    """log of the noised mixture density at x (scipy, float64)."""
    a = math.sqrt(ab[n]); s2 = ab[n] * s0 * s0 + 1.0 - ab[n]
    d2 = ((x[None, :] - a * means) ** 2).sum(axis=1)
    return logsumexp(-d2 / (2 * s2)) - math.log(len(means)) - math.log(2 * math.pi * s2)


@pytest.mark.parametrize("n", [0, 10, 55, 99])
def test_gmm_eps_is_scaled_score(n):
    tb = schedule.ddpm(100)
    means, s0 = W.gmm_components(W.WORKLOADS["gmm2d_ddpm100"].model)
    rng = np.random.default_rng(n)
    xs = rng.standard_normal((6, 2)) * 3
    eps = denoisers.gmm2d_eps(xs, np.full(6, n), tb.alphabar, means, s0, np.float64)
    h = 1e-5
    for x, e in zip(xs, eps):
        g = np.array([(_log_q(x + h * u, n, tb.alphabar, means, s0)
                       - _log_q(x - h * u, n, tb.alphabar, means, s0)) / (2 * h)
                      for u in np.eye(2)])
        assert np.allclose(e, -math.sqrt(1 - tb.alphabar[n]) * g, atol=1e-7)


def test_gmm_standard_normal_data():
    tb = schedule.ddpm(100)
    x = np.random.default_rng(0).standard_normal((5, 2))
    for n in (0, 50, 99):
        e = denoisers.gmm2d_eps(x, np.full(5, n), tb.alphabar, np.zeros((1, 2)), 1.0)
        assert np.allclose(e, math.sqrt(1 - tb.alphabar[n]) * x, rtol=1e-13)


def test_gmm_float32_close_to_float64():
    tb = schedule.ddpm(100)
    means, s0 = W.gmm_components(W.WORKLOADS["gmm2d_ddpm100"].model)
    x = np.random.default_rng(3).standard_normal((50, 2)) * 4
    n = np.arange(50) * 2
    e64 = denoisers.gmm2d_eps(x, n, tb.alphabar, means, s0, np.float64)
    e32 = denoisers.gmm2d_eps(x.astype(np.float32), n, tb.alphabar, means, s0, np.float32)
    assert e32.dtype == np.float32
    assert np.linalg.norm(e32 - e64) / np.linalg.norm(e64) < 1e-5


def test_embedding_special_values():
    e = denoisers.timestep_embedding(np.array([0, 1, 7]), 320)
    assert np.array_equal(e[0], np.r_[np.zeros(160), np.ones(160)])
    assert abs(e[1, 0] - math.sin(1.0)) < 1e-15 and abs(e[1, 160] - math.cos(1.0)) < 1e-15
    f_last = 10000.0 ** (-159 / 160)
    assert abs(e[2, 159] - math.sin(7 * f_last)) < 1e-14
    assert np.allclose((e ** 2).sum(axis=1), 160.0)


def _torch_weights(w):
    return {k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in w.items()}


def test_mlp_matches_torch_library():
    m = W.ModelSpec("mlp", (4, 5), width=64, weight_seed=3)
    w = W.make_weights(m)
    x = np.random.default_rng(0).standard_normal((7, 20))
    n = np.array([0, 3, 9, 50, 99, 1, 2])
    ours = denoisers.mlp_eps(x, n, w, 64, np.float64)
    tw = _torch_weights(w)
    emb = torch.from_numpy(denoisers.timestep_embedding(n, 64))
    h = F.gelu(F.linear(torch.from_numpy(x), tw["W1"], tw["b1"]) + emb)
    h = F.gelu(F.linear(h, tw["W2"], tw["b2"]))
    h = F.gelu(F.linear(h, tw["W3"], tw["b3"]))
    ref = F.linear(h, tw["W4"], tw["b4"]).numpy()
    assert np.allclose(ours, ref, rtol=1e-12, atol=1e-12)


def _torch_conv_stack(x, shift, tw):
    C, Wd = tw["W1"].shape[1], tw["W1"].shape[0]
    h = F.silu(F.conv2d(x, tw["W1"].view(Wd, C, 1, 1)) + shift.view(1, -1, 1, 1))
    h = F.silu(F.conv2d(h, tw["W2"].view(Wd, Wd, 1, 1), tw["b2"]))
    h = F.silu(F.conv2d(h, tw["W3"].view(Wd, Wd, 1, 1), tw["b3"]))
    return F.conv2d(h, tw["W4"].view(C, Wd, 1, 1), tw["b4"])


@pytest.mark.parametrize("cond", [0, 24])
def test_conv1x1_matches_torch_conv2d(cond):
    m = W.ModelSpec("conv1x1", (4, 6, 5), width=32, cond_dim=cond, guidance=7.5,
                    weight_seed=1, cond_seed=2)
    w = W.make_weights(m)
    x = np.random.default_rng(1).standard_normal((3, 4, 6, 5))
    n = np.array([0, 17, 999])
    ours = denoisers.conv1x1_eps(x, n, w, 32, 7.5 if cond else 1.0, np.float64)
    tw = _torch_weights(w)
    for r in range(3):
        emb = torch.from_numpy(denoisers.timestep_embedding(n[r:r + 1], 32)[0])
        xt = torch.from_numpy(x[r:r + 1])
        eu = _torch_conv_stack(xt, tw["b1"] + emb, tw)
        if cond:
            ec = _torch_conv_stack(xt, tw["b1"] + emb + tw["Wc"] @ tw["c"], tw)
            ref = eu + 7.5 * (ec - eu)
        else:
            ref = eu
        assert np.allclose(ours[r], ref[0].numpy(), rtol=1e-11, atol=1e-11)


def test_guidance_limits():
    m = W.ModelSpec("conv1x1", (4, 3, 3), width=16, cond_dim=8, weight_seed=5)
    w = W.make_weights(m)
    x = np.random.default_rng(2).standard_normal((2, 4, 3, 3))
    n = np.array([5, 40])
    e0 = denoisers.conv1x1_eps(x, n, w, 16, 0.0)
    e1 = denoisers.conv1x1_eps(x, n, w, 16, 1.0)
    wu = {k: v for k, v in w.items() if k not in ("Wc", "c")}
    eu = denoisers.conv1x1_eps(x, n, wu, 16, 1.0)
    wc = dict(wu); wc["b1"] = wc["b1"] + (w["Wc"].astype(np.float64) @ w["c"]).astype(np.float32)
    assert np.allclose(e0, eu, atol=1e-13)                 # w = 0: unconditional
    ec = denoisers.conv1x1_eps(x, n, wc, 16, 1.0)
    assert np.allclose(e1, ec, atol=1e-6)                  # w = 1: conditional


def test_bf16_rounding_matches_torch():
    v = np.random.default_rng(0).standard_normal(100_000).astype(np.float32) * 100
    v[:4] = [np.inf, -np.inf, 0.0, -0.0]
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(denoisers.bf16_round(v), ref)
    assert np.isnan(denoisers.bf16_round(np.array([np.nan], np.float32)))[0]


def test_bf16_mode_close_to_f32():
    m = W.ModelSpec("conv1x1", (4, 8, 8), width=64, weight_seed=9)
    w = W.make_weights(m)
    x = np.random.default_rng(4).standard_normal((2, 4, 8, 8)).astype(np.float32)
    n = np.array([3, 500])
    a = denoisers.conv1x1_eps(x, n, w, 64, 1.0, np.float32)
    b = denoisers.conv1x1_eps(x, n, w, 64, 1.0, np.float32, bf16=True)
    rel = np.linalg.norm(a - b) / np.linalg.norm(a)
    assert 1e-4 < rel < 2e-2
