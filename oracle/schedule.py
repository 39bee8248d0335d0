"""Noise schedules and per-step drift coefficients -- oracle side.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this.

Time runs forward for the reverse process (Sec. 2, "Notation"): reverse index
i = 0 is the prior and i = T is the sample.  The network's own (forward
diffusion) timestep for reverse step i is n_i.

DDPM (Sec. 2, the inference-model equation; Ho et al. 2020):
  beta_n  = beta_start + n * (beta_end - beta_start) / (T_train - 1)
  alpha_n = 1 - beta_n,  abar_n = prod_{m<=n} alpha_m,  abar_{-1} = 1
  n_i     = T - 1 - i    (T == T_train)
  mean    mu = (x - beta_n / sqrt(1 - abar_n) * eps) / sqrt(alpha_n)
  The Picard method consumes the *drift* "p_theta(x) - x" (Algorithm 1, drift
  line; Sec. 3, "h_t(x) - x"), here written y_i = A_i x + B_i eps with
    A_i = 1/sqrt(alpha_n) - 1,   B_i = -beta_n / (sqrt(alpha_n) sqrt(1 - abar_n)).
  sigma^2_i = beta_n (1 - abar_{n-1}) / (1 - abar_n)   (posterior variance; 0 at n = 0)

DDIM (Song et al. 2021) on the sub-chain n_i = (T-1-i) * c, c = T_train / T:
  a' = abar_{n_i - c} (1 if n_i - c < 0);  x0 = (x - sqrt(1-abar_n) eps) / sqrt(abar_n)
  s2_eta = eta^2 (1 - a')/(1 - abar_n) (1 - abar_n / a')
  x_prev = sqrt(a') x0 + sqrt(1 - a' - s2_eta) eps + sqrt(s2_eta) z
  A_i = sqrt(a' / abar_n) - 1
  B_i = sqrt(1 - a' - s2_eta) - sqrt(a' (1 - abar_n) / abar_n)
  noise variance of step i: s2_eta; tolerance variance of step i: the DDPM
  (eta = 1) value on the same sub-chain, as the footnote on the relaxed
  tolerance in Sec. 3.1 asks for ODE samplers.

Heun on the DDIM probability-flow ODE (eta = 0; Sec. 3.3: the Euler step of
Algorithm 1's drift swapped for a higher-order solver such as Heun).  In the
coordinates xbar = x / sqrt(abar), s = sqrt(1 - abar) / sqrt(abar) the ODE is
dxbar/ds = eps(x), and a DDIM step is its Euler step.  Heun's step adds the
trapezoidal correction with eps at the Euler prediction:
  x~      = x_i + (A_i x_i + B_i eps(x_i, n_i))          (the DDIM step)
  y_i     = A_i x_i + (B_i / 2) (eps(x_i, n_i) + eps(x~, n_{i+1}))
for every step but the last, whose target s = 0 has no network timestep: it
keeps the Euler (DDIM) drift, as is usual for Heun samplers.

DPM-Solver++ second-order multistep on the same eta = 0 chain (the paper's
ParaDPMSolver, Sec. 4: DPMSolver's steps solved by Picard iteration).  With
alpha = sqrt(abar), sig = sqrt(1 - abar), lambda = log(alpha / sig), the data
prediction x0 = (x - sig eps) / alpha and h_i = lambda_{i+1} - lambda_i,
r_i = h_{i-1} / h_i, phi_i = exp(-h_i) - 1:
  x_{i+1} = (sig_{i+1}/sig_i) x_i - alpha_{i+1} phi_i D_i,
  D_i = (1 + 1/(2 r_i)) x0_i - (1/(2 r_i)) x0_{i-1},
so the drift is y_i = P_i x_i + Q_i eps_i + R_i x_{i-1} + S_i eps_{i-1} with
  P_i = sig_{i+1}/sig_i - alpha_{i+1} phi_i (1 + 1/(2 r_i)) / alpha_i - 1,
  Q_i = alpha_{i+1} phi_i (1 + 1/(2 r_i)) sig_i / alpha_i,
  R_i = alpha_{i+1} phi_i / (2 r_i alpha_{i-1}),  S_i = -R_i sig_{i-1}.
The first step (no x_{i-1}) and the last (sig = 0: lambda infinite) are first
order, i.e. the DDIM step (P = A, Q = B, R = S = 0).  Tables A, B hold P, Q.

All tables are built in float64 in the order written above and rounded once to
float32 for the float32 path.  Pinned in tests/test_oracle_schedule.py (closed
forms, the DDIM(eta=1) == DDPM identity, exact recovery of a point mass).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


@dataclasses.dataclass
class Tables:
    kind: str
    T: int
    T_train: int
    model_t: np.ndarray     # int32 [T]   network timestep n_i of reverse step i
    A: np.ndarray           # float64 [T] drift coefficient on x
    B: np.ndarray           # float64 [T] drift coefficient on eps
    noise_var: np.ndarray   # float64 [T] variance of the noise z_i added by step i
    tol_var: np.ndarray     # float64 [T] sigma^2_i used by the stopping rule
    alphabar: np.ndarray    # float64 [T_train] abar_n (network timestep axis)
    solver: str = "euler"   # "euler", "heun" or "dpm2m"
    R: np.ndarray = None    # float64 [T] (dpm2m) drift coefficient on x_{i-1}
    S: np.ndarray = None    # float64 [T] (dpm2m) drift coefficient on eps_{i-1}

    @property
    def model_t_next(self) -> np.ndarray:
        """int32 [T]: network timestep of step i + 1 (-1 for the last step)."""
        out = np.empty(self.T, dtype=np.int32)
        out[:-1] = self.model_t[1:]
        out[-1] = -1
        return out

    def rs_dtype(self, dtype):
        """(R, S) rounded once to ``dtype`` (zeros unless dpm2m)."""
        z = np.zeros(self.T)
        return ((self.R if self.R is not None else z).astype(dtype),
                (self.S if self.S is not None else z).astype(dtype))

    def as_dtype(self, dtype):
        """(A, B, noise_std, tol_var) rounded once to ``dtype``."""
        return (self.A.astype(dtype), self.B.astype(dtype),
                np.sqrt(self.noise_var).astype(dtype), self.tol_var.astype(dtype))


def betas(T_train: int, beta_start: float, beta_end: float) -> np.ndarray:
    step = (beta_end - beta_start) / (T_train - 1) if T_train > 1 else 0.0
    return np.array([beta_start + n * step for n in range(T_train)], dtype=np.float64)


def alphabars(beta: np.ndarray) -> np.ndarray:
    out = np.empty_like(beta)
    acc = 1.0
    for n, b in enumerate(beta):          # sequential product, fixed order
        acc = acc * (1.0 - b)
        out[n] = acc
    return out


def ddpm(T: int, beta_start: float = 1e-4, beta_end: float = 0.02) -> Tables:
    beta = betas(T, beta_start, beta_end)
    ab = alphabars(beta)
    A = np.empty(T); Bc = np.empty(T); var = np.empty(T)
    nt = np.empty(T, dtype=np.int32)
    for i in range(T):
        n = T - 1 - i
        a = 1.0 - beta[n]
        ab_prev = ab[n - 1] if n >= 1 else 1.0
        nt[i] = n
        A[i] = 1.0 / math.sqrt(a) - 1.0
        Bc[i] = -beta[n] / (math.sqrt(a) * math.sqrt(1.0 - ab[n]))
        var[i] = beta[n] * (1.0 - ab_prev) / (1.0 - ab[n])
    return Tables("ddpm", T, T, nt, A, Bc, var, var.copy(), ab)


def ddim(T_train: int, T: int, eta: float = 0.0, beta_start: float = 1e-4,
         beta_end: float = 0.02, solver: str = "euler") -> Tables:
    if T_train % T != 0:
        raise ValueError("DDIM needs T_train to be a multiple of T")
    if solver not in ("euler", "heun", "dpm2m"):
        raise ValueError(solver)
    if solver != "euler" and eta != 0.0:
        raise ValueError("Heun and DPM-Solver integrate the eta = 0 (ODE) chain only")
    c = T_train // T
    beta = betas(T_train, beta_start, beta_end)
    ab = alphabars(beta)
    A = np.empty(T); Bc = np.empty(T); var = np.empty(T); tol = np.empty(T)
    nt = np.empty(T, dtype=np.int32)
    for i in range(T):
        n = (T - 1 - i) * c
        npv = n - c
        ap = ab[npv] if npv >= 0 else 1.0
        an = ab[n]
        v1 = (1.0 - ap) / (1.0 - an) * (1.0 - an / ap)     # eta = 1 variance
        s2 = eta * eta * v1
        nt[i] = n
        A[i] = math.sqrt(ap / an) - 1.0
        Bc[i] = math.sqrt(1.0 - ap - s2) - math.sqrt(ap * (1.0 - an) / an)
        var[i] = s2
        tol[i] = v1
    tb = Tables("ddim", T, T_train, nt, A, Bc, var, tol, ab, solver)
    if solver == "dpm2m":
        tb.R = np.zeros(T)
        tb.S = np.zeros(T)
        for i in range(1, T - 1):          # second order between the first and last steps
            n = int(nt[i])
            a, sg = math.sqrt(ab[n]), math.sqrt(1.0 - ab[n])
            a1, s1 = math.sqrt(ab[n - c]), math.sqrt(1.0 - ab[n - c])
            a0, s0 = math.sqrt(ab[n + c]), math.sqrt(1.0 - ab[n + c])
            lam, lam1, lam0 = math.log(a / sg), math.log(a1 / s1), math.log(a0 / s0)
            h, h0 = lam1 - lam, lam - lam0
            r = h0 / h
            phi = math.expm1(-h)
            g = 1.0 + 1.0 / (2.0 * r)
            A[i] = s1 / sg - a1 * phi * g / a - 1.0
            Bc[i] = a1 * phi * g * sg / a
            tb.R[i] = a1 * phi / (2.0 * r * a0)
            tb.S[i] = -tb.R[i] * s0
    return tb


def from_spec(spec) -> Tables:
    """Tables for a ``workloads.ScheduleSpec``."""
    if spec.kind == "ddpm":
        return ddpm(spec.T, spec.beta_start, spec.beta_end)
    if spec.kind == "ddim":
        return ddim(spec.T_train, spec.T, spec.eta, spec.beta_start, spec.beta_end,
                    getattr(spec, "solver", "euler"))
    raise ValueError(spec.kind)
