"""Writes the oracle's results for the full-size workloads to tests/golden/.

Calls only ``oracle`` and the seeded-input module ``workloads``; no value here
comes from the device path.  Run from the repository root:

    python tests/golden/make_golden.py [workload ...]

For every workload it stores two files:

* ``<name>.json``: the iteration count K, the stride of every iteration, the
  model evaluations and the squared norm of the sample (float64 sum of the
  float32 values);
* ``<name>.npz``: every value of the float32 sample (shape [batch, D]).

Each holds the Picard sampler's result and, where listed, the sequential
sampler's, Picard's with the sigma^2_{t+j-1} reading of the stride test, and
Picard's under Prop. 2's total-variation stopping rule.  Runs in float32 (the
device path's precision, which also decides the strides); the bf16 workload
uses the oracle's bf16-operand mode.
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import workloads as W  # noqa: E402
from oracle import Problem  # noqa: E402

SEQUENTIAL = {"gmm2d_ddpm100", "policy_mlp_ddpm100", "latent_ddpm1000_p64",
              "policy_mlp_dpm15", "latent_dpm200_p64"}
# also run with the sigma^2_{t+j-1} reading of the stride test
TOL_OFFSET_M1 = {"latent_ddpm1000_p64", "policy_mlp_ddpm100"}
# also run with Prop. 2's rule |x^{k+1} - x^k|^2 <= 4 eps^2 sigma^2 / T^2, at
# these total-variation bounds eps
PROP2_EPS = {"gmm2d_ddpm100": (1.0,), "policy_mlp_ddpm100": (1.0, 10.0)}


def summarize(x: np.ndarray) -> dict:
    flat = np.asarray(x, np.float32).reshape(-1)
    return {"norm2": float(np.sum(flat.astype(np.float64) ** 2))}


def _picard_entry(r) -> dict:
    return {"iters": r.iters, "evals": r.evals, "trace": r.trace, **summarize(r.x)}


def run(name: str):
    wl = W.WORKLOADS[name]
    weights = W.make_weights(wl.model)
    pr = Problem(wl, weights, np.float32)
    arrays = {}
    t0 = time.time()
    r = pr.picard()
    out = {"workload": name, "p": wl.p, "tau": wl.tau, "batch": wl.batch,
           "noise_seed": wl.noise_seed, "weight_seed": wl.model.weight_seed,
           "oracle_dtype": "float32" + ("+bf16-operands" if wl.model.dtype == "bf16" else ""),
           "picard": _picard_entry(r), "picard_seconds": time.time() - t0}
    arrays["picard"] = np.asarray(r.x, np.float32)
    print(name, "picard K", r.iters, "evals", r.evals, "%.1fs" % (time.time() - t0), flush=True)
    if name in TOL_OFFSET_M1:
        t0 = time.time()
        r1 = pr.picard(tol_offset=-1)
        out["picard_tol_offset_m1"] = _picard_entry(r1)
        arrays["picard_tol_offset_m1"] = np.asarray(r1.x, np.float32)
        print(name, "picard (tol_offset -1) K", r1.iters, "%.1fs" % (time.time() - t0), flush=True)
    for eps in PROP2_EPS.get(name, ()):
        t0 = time.time()
        r2 = pr.picard(tau=eps, rule="prop2")
        key = f"picard_prop2_eps{eps:g}"
        out[key] = {"eps": eps, **_picard_entry(r2)}
        arrays[key] = np.asarray(r2.x, np.float32)
        print(name, f"picard (Prop. 2, eps {eps:g}) K", r2.iters, "%.1fs" % (time.time() - t0),
              flush=True)
    if name in SEQUENTIAL:
        t0 = time.time()
        xs = pr.sequential()
        out["sequential"] = summarize(xs)
        out["sequential_seconds"] = time.time() - t0
        arrays["sequential"] = np.asarray(xs, np.float32)
        print(name, "sequential %.1fs" % (time.time() - t0), flush=True)
    return out, arrays


if __name__ == "__main__":
    names = sys.argv[1:] or list(W.WORKLOADS)
    for name in names:
        res, arrays = run(name)
        with open(os.path.join(HERE, f"{name}.json"), "w") as f:
            json.dump(res, f, indent=0)
        np.savez(os.path.join(HERE, f"{name}.npz"), **arrays)
