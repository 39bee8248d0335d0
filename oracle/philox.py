"""Philox4x32-10 and Box-Muller normals -- oracle side.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this.

Algorithm 1 draws the prior point and every step's noise up front, before
the first iteration (Sec. 3.1 and the setup of Algorithm 1).  The paper does
not name a generator; the oracle and the library fix a counter-based one so
that both draw the *same* numbers independently:

* Philox4x32-10 as defined by Salmon, Moraes, Dror and Shaw, "Parallel Random
  Numbers: As Easy as 1, 2, 3" (SC'11): a 128-bit counter, a 64-bit key, ten
  rounds of two 32x32->64-bit multiplies with the published multipliers, and a
  Weyl-sequence key schedule with the published increments.
* counter = (q mod 2^32, q div 2^32, stream, 0), key = (seed mod 2^32, seed
  div 2^32); block q yields the four 32-bit words r0..r3 for normals 4q..4q+3.
* u = (r + 0.5) * 2^-32 in float64, so u lies strictly inside (0, 1).
* Box-Muller in float64 on the pairs (u0, u1) and (u2, u3):
  n[4q]   = sqrt(-2 ln u0) cos(2 pi u1),  n[4q+1] = sqrt(-2 ln u0) sin(2 pi u1),
  n[4q+2] = sqrt(-2 ln u2) cos(2 pi u3),  n[4q+3] = sqrt(-2 ln u2) sin(2 pi u3),
  each rounded once to float32.
* stream 0 = prior point x_0 (index b*D + d); stream 1 = step noise before
  scaling (index (i*B + b)*D + d for reverse step i).

Pinned by the generator's published known-answer vectors and by moment / KS
tests of the normals (tests/test_oracle_rng.py).
"""
from __future__ import annotations

import numpy as np

# published Philox4x32 constants (Salmon et al. 2011)
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85

STREAM_PRIOR = 0
STREAM_STEP_NOISE = 1

_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(counters: np.ndarray, key: tuple[int, int]) -> np.ndarray:
    """Apply Philox4x32-10 to an (N, 4) uint32 array of counters; returns (N, 4) uint32."""
    c = np.asarray(counters, dtype=np.uint32).astype(np.uint64)
    c0, c1, c2, c3 = c[:, 0], c[:, 1], c[:, 2], c[:, 3]
    k0 = int(key[0]) & 0xFFFFFFFF
    k1 = int(key[1]) & 0xFFFFFFFF
    m0 = np.uint64(PHILOX_M0)
    m1 = np.uint64(PHILOX_M1)
    for rnd in range(10):
        if rnd > 0:                         # key schedule between rounds
            k0 = (k0 + PHILOX_W0) & 0xFFFFFFFF
            k1 = (k1 + PHILOX_W1) & 0xFFFFFFFF
        p0 = m0 * c0                        # exact: both factors < 2^32
        p1 = m1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c0, c1, c2, c3 = (hi1 ^ c1 ^ np.uint64(k0), lo1,
                          hi0 ^ c3 ^ np.uint64(k1), lo0)
    return np.stack([c0, c1, c2, c3], axis=1).astype(np.uint32)


def normals(seed: int, stream: int, count: int) -> np.ndarray:
    """Standard normals n[0..count) of one stream, float32."""
    nq = (count + 3) // 4
    q = np.arange(nq, dtype=np.uint64)
    ctr = np.zeros((nq, 4), dtype=np.uint32)
    ctr[:, 0] = (q & _MASK).astype(np.uint32)
    ctr[:, 1] = (q >> np.uint64(32)).astype(np.uint32)
    ctr[:, 2] = stream
    r = philox4x32_10(ctr, (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))
    u = (r.astype(np.float64) + 0.5) * 2.0**-32
    out = np.empty((nq, 4), dtype=np.float64)
    for a, b in ((0, 1), (2, 3)):
        rad = np.sqrt(-2.0 * np.log(u[:, a]))
        th = 2.0 * np.pi * u[:, b]
        out[:, a] = rad * np.cos(th)
        out[:, b] = rad * np.sin(th)
    return out.reshape(-1)[:count].astype(np.float32)


def prior(seed: int, batch: int, D: int) -> np.ndarray:
    """x_0 ~ N(0, I): float32 array [batch, D]."""
    return normals(seed, STREAM_PRIOR, batch * D).reshape(batch, D)


def step_normals(seed: int, T: int, batch: int, D: int) -> np.ndarray:
    """Unscaled per-step normals: float32 array [T, batch, D]."""
    return normals(seed, STREAM_STEP_NOISE, T * batch * D).reshape(T, batch, D)
