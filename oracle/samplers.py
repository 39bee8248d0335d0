"""Sequential and Picard (ParaDiGMS) samplers on full arrays -- oracle side.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this.

Notation follows the paper: time increases along the reverse process, x_0 is
the prior point and x_T the sample; y_i is the drift of step i and z_i its
up-front noise.

sequential()  -- the chain x_{i+1} = h_i(x_i) = x_i + y_i + z_i (Sec. 3, the
                 nested-function view of sequential sampling), drift form.
drifts()      -- y_i of a batch of steps: Euler (the DDPM/DDIM step), Heun's
                 step on the DDIM ODE (Sec. 3.3: any solver can supply
                 Algorithm 1's drift; two network evaluations per step, one
                 for the last), or DPM-Solver++(2M), whose drift also reads the
                 previous step's point and epsilon (Picard evaluates the point
                 before the window once per iteration for it).
sequential_mean_form() -- the same chain through the textbook step means
                 (DDPM: Ho et al.; DDIM: Song et al.), used to pin the drift
                 coefficients.
picard()      -- Algorithm 1, step for step, on the whole trajectory array:
                 drifts of the p window points in one batch, the window rebuilt
                 from its left end plus running sums of drift and noise, the
                 per-point error (1/D)|x^{k+1} - x^k|^2 over window offsets
                 [1, p), the stride = first offset whose error exceeds
                 tau^2 sigma^2 (else p), new points initialised to the window's
                 last point, t += stride, p = min(p, T - t).  With
                 ``rule="prop2"`` the stride test is Prop. 2's instead: the
                 squared norm |x^{k+1} - x^k|^2 (no 1/D) against
                 4 eps^2 sigma^2 / T^2, with the total-variation bound eps
                 passed as ``tau``.

Readings of the text that Algorithm 1 leaves open:
* the sigma in the stride test is that of the point's own absolute step,
  sigma^2_{t+j} (``tol_offset=0``); ``tol_offset=-1`` selects sigma^2_{t+j-1};
* "error > tol" fails, equality passes, and a NaN error fails;
* tol = tau^2 sigma^2, except that a step with sigma^2 = 0 (the noise-free last
  step) is always held to tol = 0, also for tau = inf (no 0 * inf);
* with a batch of several samples sharing one window, an offset fails when any
  sample fails;
* new points past T are not created (the window never extends past T);
* a non-finite point or error stops the run with ``NumericError``;
* Prop. 2's threshold factor 4 eps^2 / T^2 is formed in float64 from eps
  (taken in the run's precision) and rounded once to that precision; the
  threshold of a point is that factor times sigma^2, as for tau^2.
The running sums follow the algorithm's formula literally, left end +
cumulative drift + cumulative noise, each cumulative sum taken in order
(numpy's ``cumsum`` accumulates sequentially).
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Optional

import numpy as np


class NumericError(RuntimeError):
    pass


@dataclasses.dataclass
class PicardResult:
    x: np.ndarray             # [B, D] sample x_T
    iters: int                # K, parallel iterations
    evals: int                # network evaluations per sample (the paper's "model
                              # evaluations"): the sum of window sizes for Euler
    trace: List[int]          # stride of every iteration


def drifts(tables, A, Bc, eps_fn: Callable, rows: np.ndarray, steps: np.ndarray, prev=None):
    """Drifts y of the consecutive steps ``steps`` ([m] step indices) at the
    points ``rows`` ([m, B, D]); returns (y, network evaluations per sample,
    eps of the rows).

    Euler: y = A x + B eps(x, n_i).  Heun (DDIM ODE): with x~ = x + (A x + B
    eps), y = A x + (B/2) (eps(x, n_i) + eps(x~, n_{i+1})), except the last
    step (Euler).  DPM-Solver++(2M): y = ((A x + B eps) + R x_{i-1}) + S
    eps_{i-1} on its second-order steps, where row 0 takes x_{i-1}, eps_{i-1}
    from ``prev`` = (x, eps) of the step before ``steps[0]``."""
    m, Bn, D = rows.shape
    e = eps_fn(rows.reshape(m * Bn, D), np.repeat(tables.model_t[steps], Bn)).reshape(m, Bn, D)
    y = A[steps, None, None] * rows + Bc[steps, None, None] * e
    if tables.solver == "dpm2m":
        R, S = tables.rs_dtype(Bc.dtype)
        for j, i in enumerate(steps):
            if R[i] == 0:
                continue                      # first-order step
            xp, ep = (rows[j - 1], e[j - 1]) if j > 0 else prev
            y[j] = (y[j] + R[i] * xp) + S[i] * ep
        return y, m, e
    if tables.solver != "heun":
        return y, m, e
    inner = steps < tables.T - 1
    if np.any(inner):
        s = steps[inner]
        r = rows[inner]
        xt = r + y[inner]
        e2 = eps_fn(xt.reshape(-1, D), np.repeat(tables.model_t_next[s], Bn)).reshape(r.shape)
        Bh = (Bc[s] * Bc.dtype.type(0.5))[:, None, None]
        y[inner] = A[s, None, None] * r + Bh * (e[inner] + e2)
    return y, m + int(np.count_nonzero(inner)), e


def stride_from_errors(err: np.ndarray, tol: np.ndarray, p_eff: int) -> int:
    """Algorithm 1's stride rule.

    err: [p_eff, B] errors (row 0 unused); tol: [p_eff] thresholds.
    Returns the smallest j in [1, p_eff) whose error fails for any sample,
    else p_eff.  A NaN error fails (the comparison is ``not err <= tol``).
    """
    for j in range(1, p_eff):
        if np.any(~(err[j] <= tol[j])):
            return j
    return p_eff


def _tables(tables, dtype):
    A, Bc, zstd, tolv = tables.as_dtype(dtype)
    return A, Bc, zstd, tolv


def make_noise(tables, normals: np.ndarray, dtype) -> np.ndarray:
    """z_i = sigma_i * n_i with sigma_i rounded to ``dtype``: [T, B, D]."""
    _, _, zstd, _ = _tables(tables, dtype)
    return zstd[:, None, None] * np.asarray(normals, dtype=dtype)


def sequential(tables, eps_fn: Callable, x0: np.ndarray, noise: np.ndarray,
               dtype=np.float32) -> np.ndarray:
    """x_{i+1} = x_i + (A_i x_i + B_i eps(x_i, n_i)) + z_i for i in [0, T)."""
    A, Bc, _, _ = _tables(tables, dtype)
    x = np.asarray(x0, dtype=dtype).copy()
    B = x.shape[0]
    prev = None
    for i in range(tables.T):
        y, _, e = drifts(tables, A, Bc, eps_fn, x[None], np.array([i]), prev)
        prev = (x, e[0])
        x = x + y[0] + noise[i]
        if not np.all(np.isfinite(x)):
            raise NumericError(f"non-finite state at step {i}")
    return x


def sequential_mean_form(tables, eps_fn: Callable, x0: np.ndarray,
                         noise: np.ndarray) -> np.ndarray:
    """Float64 chain through the textbook step means, for pinning A_i and B_i."""
    x = np.asarray(x0, dtype=np.float64).copy()
    B = x.shape[0]
    ab = tables.alphabar
    c = tables.T_train // tables.T
    for i in range(tables.T):
        n = int(tables.model_t[i])
        e = eps_fn(x, np.full(B, n))
        if tables.kind == "ddpm":
            beta = 1.0 - ab[n] / (ab[n - 1] if n >= 1 else 1.0)
            mu = (x - beta / np.sqrt(1.0 - ab[n]) * e) / np.sqrt(1.0 - beta)
        else:
            ap = ab[n - c] if n - c >= 0 else 1.0
            s2 = tables.noise_var[i]
            x0p = (x - np.sqrt(1.0 - ab[n]) * e) / np.sqrt(ab[n])
            mu = np.sqrt(ap) * x0p + np.sqrt(1.0 - ap - s2) * e
        x = mu + noise[i]
    return x


RULES = ("relaxed", "prop2")


def stop_factor(rule: str, tau: float, T: int, dtype) -> np.floating:
    """Factor of sigma^2 in the stride test's threshold: tau^2 for the relaxed
    rule of Sec. 3.1 (per-dimension mean error), 4 eps^2 / T^2 for Prop. 2
    (squared norm; eps = ``tau``)."""
    f = np.dtype(dtype).type
    t = f(tau)
    if rule == "relaxed":
        return t * t
    if rule == "prop2":
        e = float(t)
        return f(4.0 * e * e / (float(T) * float(T)))
    raise ValueError(f"unknown stopping rule {rule!r}")


def picard(tables, eps_fn: Callable, x0: np.ndarray, noise: np.ndarray,
           p: int, tau: float, dtype=np.float32, tol_offset: int = 0,
           on_iter: Optional[Callable] = None, rule: str = "relaxed") -> PicardResult:
    """Algorithm 1 on a full [T+1, B, D] trajectory array.

    x0: [B, D] prior point; noise: [T, B, D] the up-front z_i.
    rule: "relaxed" (Sec. 3.1: (1/D)|dx|^2 <= tau^2 sigma^2) or "prop2"
    (Prop. 2: |dx|^2 <= 4 tau^2 sigma^2 / T^2, tau being the bound eps).
    ``on_iter(k, t, p_eff, x_old, x_new, err, stride)`` is called after each
    iteration, for tests: x_old[j] is x^k_{t+j} for j in [0, p_eff] and
    x_new[j] is x^{k+1}_{t+j+1} for j in [0, p_eff).
    """
    T = tables.T
    A, Bc, _, tolv = _tables(tables, dtype)
    tau2 = stop_factor(rule, tau, T, dtype)
    x0 = np.asarray(x0, dtype=dtype)
    Bn, D = x0.shape
    X = np.empty((T + 1, Bn, D), dtype=dtype)
    t, k, evals = 0, 0, 0
    pe = min(p, T)
    X[0] = x0                                   # prior point
    X[1:pe + 1] = x0                            # initial window = copies of x_0
    trace: List[int] = []
    while t < T:
        rows = X[t:t + pe]                      # x^k_{t+j}, j in [0, pe)
        prev, nh = None, 0
        if tables.solver == "dpm2m" and t >= 1:  # the multistep drift needs x_{t-1}, eps_{t-1}
            eh = eps_fn(X[t - 1], np.full(Bn, tables.model_t[t - 1]))
            prev, nh = (X[t - 1], eh), 1
        Y, nev, _ = drifts(tables, A, Bc, eps_fn, rows, np.arange(t, t + pe), prev)
        nev += nh
        Xn = X[t] + np.cumsum(Y, axis=0) + np.cumsum(noise[t:t + pe], axis=0)
        if not np.all(np.isfinite(Xn)):
            raise NumericError(f"non-finite window at iteration {k}")
        err = np.zeros((pe, Bn), dtype=dtype)
        tol = np.zeros(pe, dtype=dtype)
        for j in range(1, pe):
            dlt = Xn[j - 1] - X[t + j]          # x^{k+1}_{t+j} - x^k_{t+j}
            if rule == "prop2":
                err[j] = np.sum(dlt * dlt, axis=1, dtype=dtype)
            else:
                err[j] = np.mean(dlt * dlt, axis=1, dtype=dtype)
            s2 = tolv[t + j + tol_offset]
            tol[j] = tau2 * s2 if s2 != 0 else s2
        if not np.all(np.isfinite(err)):
            raise NumericError(f"non-finite error at iteration {k}")
        stride = stride_from_errors(err, tol, pe)
        x_old = X[t:t + pe + 1].copy() if on_iter is not None else None
        X[t + 1:t + pe + 1] = Xn
        hi = min(t + pe + stride, T)
        if hi > t + pe:
            X[t + pe + 1:hi + 1] = X[t + pe]    # new points = window's last point
        if on_iter is not None:
            on_iter(k, t, pe, x_old, Xn, err, stride)
        evals += nev
        trace.append(stride)
        t += stride
        k += 1
        pe = min(p, T - t)
    return PicardResult(X[T].copy(), k, evals, trace)
