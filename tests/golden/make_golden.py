"""Writes the oracle's results for the full-size workloads to tests/golden/.

Calls only ``oracle`` and the seeded-input module ``workloads``; no value here
comes from the device path.  Run from the repository root:

    python tests/golden/make_golden.py [workload ...]

For every workload it stores, as JSON: the iteration count K, the stride of
every iteration, the model evaluations, the squared norm of the sample (float64
sum of the float32 values) and the sample's values at 4096 fixed indices
(every index for samples smaller than that), for the Picard sampler and, where
listed, for the sequential sampler and for Picard with the sigma^2_{t+j-1}
reading of the stride test.  Runs in float32 (the device path's
precision, which also decides the strides); the bf16 workload uses the
oracle's bf16-operand mode.
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

N_SAMPLE = 4096
SEQUENTIAL = {"gmm2d_ddpm100", "policy_mlp_ddpm100", "latent_ddpm1000_p64",
              "policy_mlp_dpm15", "latent_dpm200_p64"}
# also run with the sigma^2_{t+j-1} reading of the stride test
TOL_OFFSET_M1 = {"latent_ddpm1000_p64", "policy_mlp_ddpm100"}


def sample_indices(n: int) -> np.ndarray:
    if n <= N_SAMPLE:
        return np.arange(n)
    return np.linspace(0, n - 1, N_SAMPLE).round().astype(np.int64)


def summarize(x: np.ndarray) -> dict:
    flat = np.asarray(x, np.float32).reshape(-1)
    idx = sample_indices(flat.size)
    return {"norm2": float(np.sum(flat.astype(np.float64) ** 2)),
            "idx": idx.tolist(), "values": [float(v) for v in flat[idx]]}


def run(name: str) -> dict:
    wl = W.WORKLOADS[name]
    weights = W.make_weights(wl.model)
    pr = Problem(wl, weights, np.float32)
    t0 = time.time()
    r = pr.picard()
    out = {"workload": name, "p": wl.p, "tau": wl.tau, "batch": wl.batch,
           "noise_seed": wl.noise_seed, "weight_seed": wl.model.weight_seed,
           "oracle_dtype": "float32" + ("+bf16-operands" if wl.model.dtype == "bf16" else ""),
           "picard": {"iters": r.iters, "evals": r.evals, "trace": r.trace, **summarize(r.x)},
           "picard_seconds": time.time() - t0}
    print(name, "picard K", r.iters, "evals", r.evals, "%.1fs" % (time.time() - t0), flush=True)
    if name in TOL_OFFSET_M1:
        t0 = time.time()
        r1 = pr.picard(tol_offset=-1)
        out["picard_tol_offset_m1"] = {"iters": r1.iters, "evals": r1.evals, "trace": r1.trace,
                                       **summarize(r1.x)}
        print(name, "picard (tol_offset -1) K", r1.iters, "%.1fs" % (time.time() - t0), flush=True)
    if name in SEQUENTIAL:
        t0 = time.time()
        xs = pr.sequential()
        out["sequential"] = summarize(xs)
        out["sequential_seconds"] = time.time() - t0
        print(name, "sequential %.1fs" % (time.time() - t0), flush=True)
    return out


if __name__ == "__main__":
    names = sys.argv[1:] or list(W.WORKLOADS)
    for name in names:
        res = run(name)
        with open(os.path.join(HERE, f"{name}.json"), "w") as f:
            json.dump(res, f, indent=0)
