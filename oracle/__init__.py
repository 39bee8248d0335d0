"""CPU oracle for the ParaDiGMS hot path (Shih et al., arXiv 2305.16317).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import anything under
``oracle/``.  The product path (``paper_2305_16317_amd`` and its HIP library)
never imports, calls or links it, and the oracle imports nothing from the
product path.  The two share only the seeded-input module ``workloads``,
which holds no arithmetic of the method.

Plain, slow NumPy, dtype-generic: float64 for the pins, float32 where a
result must be compared with the float32 device path, because the stride of
every iteration is an integer decided by floating-point comparisons and both
sides must take that decision in the same precision.

Modules
  philox     -- Philox4x32-10 + Box-Muller (the up-front noise of Algorithm 1)
  schedule   -- DDPM / DDIM coefficient tables (Sec. 2)
  denoisers  -- synthetic epsilon-predictors standing in for the paper's networks
  samplers   -- sequential chain and Algorithm 1 on full arrays

Pins (tests/test_oracle_*.py):
  philox     published known-answer vectors; normal moments and KS test
  schedule   closed forms; DDIM(eta=1, T=T_train) == DDPM; exact recovery
             of a point mass by both samplers
  denoisers  mixture score vs finite differences of the log-density;
             layer stacks vs PyTorch CPU library routines; guidance limits
  samplers   p = 1 equals the sequential chain bitwise; tau = 0 equals it;
             tau = inf has a closed form; K <= T and the first k points are
             exact after k iterations (Prop. 1 and the remark after it);
             the linear-Gaussian error recursion; brute force for T <= 4
Parity unpinned: the iteration counts K and final samples of the five full
workloads have no value printed in the paper; they are pinned only through
the properties above and compared device-vs-oracle.
"""
from __future__ import annotations

import numpy as np

from . import denoisers, philox, samplers, schedule

__all__ = ["philox", "schedule", "denoisers", "samplers", "Problem"]


class Problem:
    """Everything the oracle needs for one workload, in one precision."""

    def __init__(self, workload, weights: dict, dtype=np.float32, bf16=None):
        self.w = workload
        self.dtype = dtype
        self.tables = schedule.from_spec(workload.schedule)
        self.weights = weights
        self.eps = denoisers.Denoiser(workload.model, weights,
                                      self.tables.alphabar, dtype, bf16)
        D = workload.model.D
        self.D = D
        self.x0 = philox.prior(workload.noise_seed, workload.batch, D).astype(dtype)
        if np.any(self.tables.noise_var > 0):
            n = philox.step_normals(workload.noise_seed, self.tables.T,
                                    workload.batch, D)
            self.noise = samplers.make_noise(self.tables, n, dtype)
        else:
            self.noise = np.zeros((self.tables.T, workload.batch, D), dtype=dtype)

    def sequential(self):
        return samplers.sequential(self.tables, self.eps, self.x0, self.noise,
                                   self.dtype)

    def picard(self, p=None, tau=None, tol_offset=0, on_iter=None, rule="relaxed"):
        return samplers.picard(self.tables, self.eps, self.x0, self.noise,
                               self.w.p if p is None else p,
                               self.w.tau if tau is None else tau,
                               self.dtype, tol_offset, on_iter, rule)
