"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module holds no arithmetic of the sampling method.  It only names the
workloads (shapes, step counts, window, tolerance, seeds) and draws the
random *inputs* that both sides are handed: denoiser weights, biases and the
conditioning vector.  The noise that the method itself draws (the prior point
and the per-step noise of the up-front sampling step of Algorithm 1) is not
made here: each side implements the Philox4x32-10 generator on its own.

Weights use numpy's Philox bit generator through its raw 64-bit output only
(``random_raw``), so the values depend on no version-specific ``Generator``
method.  Xavier-uniform weights (Glorot & Bengio 2010) and the usual
``U(-1/sqrt(fan_in), 1/sqrt(fan_in))`` biases stand in for trained weights,
which the paper's experiments use but which are not available here.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Tuple

import numpy as np

__all__ = [
    "ScheduleSpec", "ModelSpec", "Workload", "WORKLOADS", "small_variant",
    "make_weights", "gmm_components", "uniform01", "std_normal",
]


@dataclasses.dataclass(frozen=True)
class ScheduleSpec:
    kind: str            # "ddpm" or "ddim"
    T_train: int         # length of the training chain (beta table length)
    T: int               # number of sampling steps
    beta_start: float = 1e-4
    beta_end: float = 0.02
    eta: float = 0.0     # DDIM only
    solver: str = "euler"  # "euler"; "heun" or "dpm2m" (DDIM with eta = 0 only)


@dataclasses.dataclass(frozen=True)
class ModelSpec:
    kind: str                          # "gmm2d", "mlp" or "conv1x1"
    sample_shape: Tuple[int, ...]
    width: int = 0                     # hidden width (mlp: 1024, conv1x1: 320)
    dtype: str = "f32"                 # GEMM operand type: "f32" or "bf16"
    cond_dim: int = 0                  # 0: unconditional; else classifier-free guidance
    guidance: float = 1.0              # guidance scale w
    weight_seed: int = 0
    cond_seed: int = 0
    # Gaussian-mixture data (gmm2d only)
    n_components: int = 8
    radius: float = 4.0
    sigma0: float = 0.3

    @property
    def D(self) -> int:
        return int(np.prod(self.sample_shape))


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    schedule: ScheduleSpec
    model: ModelSpec
    p: int
    tau: float
    batch: int = 1
    noise_seed: int = 0


_DDPM100 = ScheduleSpec("ddpm", 100, 100)
_DDPM1000 = ScheduleSpec("ddpm", 1000, 1000)
_DDIM200 = ScheduleSpec("ddim", 1000, 200, eta=0.0)
_LATENT = (4, 96, 96)

WORKLOADS: Dict[str, Workload] = {
    # 8-component 2-D Gaussian mixture with its exact score
    "gmm2d_ddpm100": Workload(
        "gmm2d_ddpm100", _DDPM100, ModelSpec("gmm2d", (2,)), p=100, tau=0.1),
    # action trajectory 16x10, 4-layer MLP of width 1024
    "policy_mlp_ddpm100": Workload(
        "policy_mlp_ddpm100", _DDPM100, ModelSpec("mlp", (16, 10), width=1024),
        p=100, tau=0.1),
    # 4x96x96 latent, per-pixel 4-320-320-320-4 stack, 1000-step DDPM
    "latent_ddpm1000_p64": Workload(
        "latent_ddpm1000_p64", _DDPM1000, ModelSpec("conv1x1", _LATENT, width=320),
        p=64, tau=0.1),
    # same network, 200-step DDIM (eta=0), four samples sharing one window
    "latent_ddim200_b4": Workload(
        "latent_ddim200_b4", _DDIM200, ModelSpec("conv1x1", _LATENT, width=320),
        p=64, tau=0.05, batch=4),
    # same network in bf16 with classifier-free guidance w=7.5, 768-d condition
    "latent_cfg_bf16_ddpm1000_p128": Workload(
        "latent_cfg_bf16_ddpm1000_p128", _DDPM1000,
        ModelSpec("conv1x1", _LATENT, width=320, dtype="bf16", cond_dim=768,
                  guidance=7.5),
        p=128, tau=0.1),
    # Heun's method on the DDIM ODE (a higher-order solver, Sec. 3.3): the
    # 16x10 policy at 20 steps, and the 4x96x96 latent at 100 steps
    "policy_mlp_heun20": Workload(
        "policy_mlp_heun20", ScheduleSpec("ddim", 100, 20, solver="heun"),
        ModelSpec("mlp", (16, 10), width=1024), p=20, tau=0.1),
    "latent_heun100_p32": Workload(
        "latent_heun100_p32", ScheduleSpec("ddim", 1000, 100, solver="heun"),
        ModelSpec("conv1x1", _LATENT, width=320), p=32, tau=0.05),
    # DPM-Solver++(2M) (ParaDPMSolver, Sec. 4): the 16x10 policy at 15 steps
    # (T_train = 90 gives the 6-apart timesteps that 15 of 100 steps take), and
    # the 4x96x96 latent at 200 steps with tau = 0.1
    "policy_mlp_dpm15": Workload(
        "policy_mlp_dpm15", ScheduleSpec("ddim", 90, 15, solver="dpm2m"),
        ModelSpec("mlp", (16, 10), width=1024), p=15, tau=0.1),
    "latent_dpm200_p64": Workload(
        "latent_dpm200_p64", ScheduleSpec("ddim", 1000, 200, solver="dpm2m"),
        ModelSpec("conv1x1", _LATENT, width=320), p=64, tau=0.1),
}


def small_variant(name: str, *, T: int | None = None, p: int | None = None,
                  shape: Tuple[int, ...] | None = None, width: int | None = None,
                  batch: int | None = None, tau: float | None = None,
                  n_components: int | None = None) -> Workload:
    """A reduced copy of a named workload (for tests the oracle finishes fast)."""
    w = WORKLOADS[name]
    s = w.schedule
    if T is not None:
        T_train = T if s.kind == "ddpm" else T * max(1, s.T_train // s.T)
        s = dataclasses.replace(s, T=T, T_train=T_train)
    m = w.model
    if shape is not None:
        m = dataclasses.replace(m, sample_shape=tuple(shape))
    if width is not None:
        m = dataclasses.replace(m, width=width)
    if n_components is not None:
        m = dataclasses.replace(m, n_components=n_components)
    return dataclasses.replace(
        w, name=w.name + "_small", schedule=s, model=m,
        p=w.p if p is None else p, tau=w.tau if tau is None else tau,
        batch=w.batch if batch is None else batch)


# ----------------------------------------------------------------------------
# random inputs

def _raw(seed: int, stream: int, n: int) -> np.ndarray:
    bg = np.random.Philox(key=np.array([seed & (2**64 - 1), stream], dtype=np.uint64))
    return bg.random_raw(n).astype(np.uint64)


def uniform01(seed: int, stream: int, n: int) -> np.ndarray:
    """n doubles in [0, 1) from the top 53 bits of raw 64-bit draws."""
    return (_raw(seed, stream, n) >> np.uint64(11)).astype(np.float64) * 2.0**-53


def std_normal(seed: int, stream: int, n: int) -> np.ndarray:
    """n standard normals (Box-Muller on raw draws), float64."""
    m = (n + 1) // 2
    u = uniform01(seed, stream, 2 * m)
    u1 = 1.0 - u[0::2]                      # (0, 1]
    r = np.sqrt(-2.0 * np.log(u1))
    th = 2.0 * np.pi * u[1::2]
    out = np.empty(2 * m)
    out[0::2] = r * np.cos(th)
    out[1::2] = r * np.sin(th)
    return out[:n]


def _xavier(seed: int, stream: int, fan_out: int, fan_in: int) -> np.ndarray:
    a = math.sqrt(6.0 / (fan_in + fan_out))
    u = uniform01(seed, stream, fan_out * fan_in)
    return (a * (2.0 * u - 1.0)).reshape(fan_out, fan_in).astype(np.float32)


def _bias(seed: int, stream: int, fan_out: int, fan_in: int) -> np.ndarray:
    a = 1.0 / math.sqrt(fan_in)
    return (a * (2.0 * uniform01(seed, stream, fan_out) - 1.0)).astype(np.float32)


def layer_dims(model: ModelSpec) -> Tuple[int, ...]:
    if model.kind == "mlp":
        return (model.D, model.width, model.width, model.width, model.D)
    if model.kind == "conv1x1":
        c = model.sample_shape[0]
        return (c, model.width, model.width, model.width, c)
    raise ValueError(model.kind)


def gmm_components(model: ModelSpec) -> Tuple[np.ndarray, float]:
    """Means on a circle of the given radius (K x 2, float64) and the shared std."""
    k = np.arange(model.n_components, dtype=np.float64)
    ang = 2.0 * np.pi * k / model.n_components
    means = model.radius * np.stack([np.cos(ang), np.sin(ang)], axis=1)
    return means, float(model.sigma0)


def make_weights(model: ModelSpec) -> Dict[str, np.ndarray]:
    """Seeded weights for a model, float32, in (out, in) layout.

    Keys: W1..W4, b1..b4 for "mlp" and "conv1x1"; additionally Wc (width x
    cond_dim) and c (cond_dim) when cond_dim > 0; "means" (K x 2) and "sigma0"
    (shape (1,)) for "gmm2d".
    """
    if model.kind == "gmm2d":
        means, s0 = gmm_components(model)
        return {"means": means.astype(np.float32),
                "sigma0": np.array([s0], dtype=np.float32)}
    dims = layer_dims(model)
    w: Dict[str, np.ndarray] = {}
    for li in range(4):
        fi, fo = dims[li], dims[li + 1]
        w[f"W{li+1}"] = _xavier(model.weight_seed, 10 + li, fo, fi)
        w[f"b{li+1}"] = _bias(model.weight_seed, 20 + li, fo, fi)
    if model.cond_dim:
        w["Wc"] = _xavier(model.weight_seed, 30, model.width, model.cond_dim)
        w["c"] = std_normal(model.cond_seed, 31, model.cond_dim).astype(np.float32)
    return w
