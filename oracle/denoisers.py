"""Synthetic denoisers eps(x, n) -- oracle side.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this.

The paper treats the network as a given oracle for the drift (Sec. 2, "we
have access to an oracle that computes the drift").  Its trained networks are
not available, so three synthetic stand-ins with the shapes of its workloads
are defined here; each is an epsilon-predictor eps(x, n) for network
timestep n.

* gmm2d: data = equal-weight mixture of K isotropic Gaussians N(mu_k, s0^2 I)
  in 2-D.  Under the forward process the marginal at step n is the mixture of
  N(a mu_k, s^2 I) with a = sqrt(abar_n), s^2 = abar_n s0^2 + 1 - abar_n, and
  the exact epsilon is -sqrt(1 - abar_n) grad log q_n(x)
  = sqrt(1 - abar_n) / s^2 * (x - a sum_k w_k mu_k),
  w = softmax_k(-|x - a mu_k|^2 / (2 s^2)).
* mlp: x in R^D (D = 160 for a 16x10 action trajectory);
  h1 = GELU(W1 x + (b1 + e_n)), h2 = GELU(W2 h1 + b2), h3 = GELU(W3 h2 + b3),
  eps = W4 h3 + b4, GELU(u) = u/2 (1 + erf(u / sqrt 2)).
* conv1x1: x in R^{C x H x W}; the same four layers applied to every pixel's
  C-vector (a stack of 1x1 convolutions) with SiLU(u) = u / (1 + exp(-u)).
  With classifier-free guidance (cond_dim > 0) the first-layer shift is
  b1 + e_n + Wc c for the conditional branch and b1 + e_n for the
  unconditional one, and eps = eps_u + w (eps_c - eps_u) (Ho & Salimans 2022;
  the paper's Table 4 uses w = 7.5).
* e_n is the sinusoidal embedding of width `width`: sin(n f_k) for k < half,
  cos(n f_{k-half}) after, f_k = exp(-ln(10^4) k / half), built in float64.

``dtype`` selects the arithmetic: float64 for pinning, float32 for parity with
the float32 device path.  ``bf16=True`` additionally rounds every matmul
operand (weights and activations) to bfloat16 with round-to-nearest-even, the
operand precision of the bf16 device path; accumulation stays in ``dtype``.
Pinned in tests/test_oracle_denoisers.py against finite differences of the
mixture log-density and against PyTorch CPU library routines.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf as _erf


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    out = r.astype(np.uint32).view(np.float32)
    return np.where(np.isnan(a), a, out)


def timestep_embedding(n: np.ndarray, dim: int, dtype=np.float64) -> np.ndarray:
    half = dim // 2
    k = np.arange(half, dtype=np.float64)
    freqs = np.exp(-math.log(10000.0) * k / half)
    args = np.asarray(n, dtype=np.float64)[:, None] * freqs[None, :]
    return np.concatenate([np.sin(args), np.cos(args)], axis=1).astype(dtype)


# ----------------------------------------------------------------------------
def gmm2d_eps(x: np.ndarray, n: np.ndarray, alphabar: np.ndarray,
              means: np.ndarray, sigma0: float, dtype=np.float64) -> np.ndarray:
    """Exact epsilon of a Gaussian mixture.  x: [M, 2]; n: [M] network timesteps."""
    x = np.asarray(x, dtype=dtype)
    ab = alphabar[np.asarray(n)]                              # float64 [M]
    a = np.sqrt(ab).astype(dtype)[:, None]
    s2_64 = ab * float(sigma0) ** 2 + 1.0 - ab
    inv2s2 = (1.0 / (2.0 * s2_64)).astype(dtype)[:, None]
    coef = (np.sqrt(1.0 - ab) / s2_64).astype(dtype)[:, None]
    mu = np.asarray(means, dtype=dtype)                       # [K, 2]
    d = x[:, None, :] - a[:, :, None] * mu[None, :, :]        # [M, K, 2]
    logits = -(d * d).sum(axis=2) * inv2s2                   # [M, K]
    logits = logits - logits.max(axis=1, keepdims=True)
    w = np.exp(logits)
    w = w / w.sum(axis=1, keepdims=True)
    mbar = w @ mu                                             # [M, 2]
    return coef * (x - a * mbar)


# ----------------------------------------------------------------------------
def _mm(h: np.ndarray, W: np.ndarray, bf16: bool) -> np.ndarray:
    if bf16:
        return bf16_round(h) @ bf16_round(W).T
    return h @ W.T


def gelu(u: np.ndarray) -> np.ndarray:
    return (0.5 * u * (1.0 + _erf(u / math.sqrt(2.0)))).astype(u.dtype)


def silu(u: np.ndarray) -> np.ndarray:
    one = u.dtype.type(1.0)
    return u / (one + np.exp(-u))


def mlp_eps(x: np.ndarray, n: np.ndarray, w: dict, width: int,
            dtype=np.float64, bf16: bool = False) -> np.ndarray:
    """x: [M, D]; n: [M]."""
    W = {k: np.asarray(v, dtype=dtype) for k, v in w.items()}
    h = np.asarray(x, dtype=dtype)
    shift = W["b1"][None, :] + timestep_embedding(n, width, dtype)
    h = gelu(_mm(h, W["W1"], bf16) + shift)
    h = gelu(_mm(h, W["W2"], bf16) + W["b2"])
    h = gelu(_mm(h, W["W3"], bf16) + W["b3"])
    return _mm(h, W["W4"], bf16) + W["b4"]


def _pixel_stack(xp: np.ndarray, shift: np.ndarray, W: dict, bf16: bool) -> np.ndarray:
    """xp: [P, C] pixel vectors of one image; shift: [width]."""
    h = silu(_mm(xp, W["W1"], bf16) + shift)
    h = silu(_mm(h, W["W2"], bf16) + W["b2"])
    h = silu(_mm(h, W["W3"], bf16) + W["b3"])
    return _mm(h, W["W4"], bf16) + W["b4"]


def conv1x1_shifts(n: int, w: dict, width: int, dtype=np.float64):
    """(unconditional, conditional-or-None) first-layer shifts for timestep n."""
    W = {k: np.asarray(v, dtype=dtype) for k, v in w.items()}
    e = timestep_embedding(np.array([n]), width, dtype)[0]
    s_u = W["b1"] + e
    s_c = None
    if "Wc" in W:
        s_c = s_u + W["Wc"] @ W["c"]
    return s_u, s_c


def conv1x1_eps(x: np.ndarray, n: np.ndarray, w: dict, width: int,
                guidance: float = 1.0, dtype=np.float64,
                bf16: bool = False) -> np.ndarray:
    """x: [M, C, H, W] (or [M, C*H*W]); n: [M].  Row by row, pixel by pixel."""
    x = np.asarray(x, dtype=dtype)
    M = x.shape[0]
    C = w["W1"].shape[1]
    xr = x.reshape(M, C, -1)
    W = {k: np.asarray(v, dtype=dtype) for k, v in w.items()}
    gw = np.dtype(dtype).type(guidance)
    out = np.empty_like(xr)
    for m in range(M):
        xp = xr[m].T                                        # [P, C]
        s_u, s_c = conv1x1_shifts(int(n[m]), w, width, dtype)
        e_u = _pixel_stack(xp, s_u, W, bf16)
        if s_c is None:
            e = e_u
        else:
            e_c = _pixel_stack(xp, s_c, W, bf16)
            e = e_u + gw * (e_c - e_u)
        out[m] = e.T
    return out.reshape(x.shape)


# ----------------------------------------------------------------------------
class Denoiser:
    """eps(x_rows, n_rows) for a ``workloads.ModelSpec`` in a chosen precision."""

    def __init__(self, model, weights: dict, alphabar: np.ndarray,
                 dtype=np.float32, bf16: bool | None = None):
        self.model = model
        self.w = weights
        self.alphabar = alphabar
        self.dtype = dtype
        self.bf16 = (model.dtype == "bf16") if bf16 is None else bf16

    def __call__(self, x: np.ndarray, n: np.ndarray) -> np.ndarray:
        m = self.model
        if m.kind == "gmm2d":
            return gmm2d_eps(x, n, self.alphabar, self.w["means"],
                             float(self.w["sigma0"][0]), self.dtype)
        if m.kind == "mlp":
            return mlp_eps(x, n, self.w, m.width, self.dtype, self.bf16)
        if m.kind == "conv1x1":
            g = m.guidance if m.cond_dim else 1.0
            return conv1x1_eps(x, n, self.w, m.width, g, self.dtype, self.bf16)
        raise ValueError(m.kind)
