"""Pins for the oracle's Philox4x32-10 + Box-Muller generator."""
import numpy as np
import pytest
from scipy import stats

from oracle import philox


# Known-answer vectors published with the Philox generator (Salmon et al.,
# SC'11, Random123 distribution): (counter, key) -> output, all 32-bit words.
KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,expect", KAT)
def test_philox_known_answers(ctr, key, expect):
    out = philox.philox4x32_10(np.array([ctr], dtype=np.uint32), key)[0]
    assert tuple(int(v) for v in out) == expect


def test_philox_vectorised_rows_independent():
    ctr = np.array([KAT[0][0], KAT[2][0], KAT[0][0]], dtype=np.uint32)
    out = philox.philox4x32_10(ctr, (0, 0))
    assert tuple(int(v) for v in out[0]) == KAT[0][2]
    assert np.array_equal(out[0], out[2])


def test_normals_moments_and_ks():
    n = philox.normals(seed=7, stream=1, count=400_000).astype(np.float64)
    assert abs(n.mean()) < 0.01
    assert abs(n.var() - 1.0) < 0.01
    assert abs(stats.kurtosis(n, fisher=False) - 3.0) < 0.05
    assert stats.kstest(n, "norm").pvalue > 1e-3


def test_streams_seeds_and_prefix_consistency():
    a = philox.normals(3, 0, 1001)
    b = philox.normals(3, 0, 17)
    assert np.array_equal(a[:17], b)                 # ragged count = prefix
    assert not np.array_equal(philox.normals(3, 1, 17), b)
    assert not np.array_equal(philox.normals(4, 0, 17), b)
    hi = philox.normals(3 + (1 << 32), 0, 17)        # high key word matters
    assert not np.array_equal(hi, b)


def test_box_muller_first_block_by_hand():
    # block 0 of seed 0 stream 0 is the first known-answer vector
    r = np.array(KAT[0][2], dtype=np.float64)
    u = (r + 0.5) / 2.0**32
    rad0 = np.sqrt(-2 * np.log(u[0])); rad2 = np.sqrt(-2 * np.log(u[2]))
    expect = np.array([rad0 * np.cos(2 * np.pi * u[1]), rad0 * np.sin(2 * np.pi * u[1]),
                       rad2 * np.cos(2 * np.pi * u[3]), rad2 * np.sin(2 * np.pi * u[3])],
                      dtype=np.float32)
    assert np.array_equal(philox.normals(0, 0, 4), expect)


def test_layouts():
    x0 = philox.prior(5, 3, 10)
    assert x0.shape == (3, 10)
    assert np.array_equal(x0.reshape(-1), philox.normals(5, philox.STREAM_PRIOR, 30))
    z = philox.step_normals(5, 4, 3, 10)
    assert z.shape == (4, 3, 10)
    flat = philox.normals(5, philox.STREAM_STEP_NOISE, 120)
    assert np.array_equal(z[2, 1], flat[(2 * 3 + 1) * 10:(2 * 3 + 2) * 10])
