"""Pins for the oracle's Gaussian noise (Section 4.3, Eq. value-perturbation).

Philox4x32-10 is pinned by the published known-answer vectors; the uniform map by
its exact end points; Box-Muller by the moments and the distribution of its output.
"""
import os

import numpy as np
import pytest
from scipy import stats

from oracle import philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            v = line.split()
            assert v[0] == "10"
            nums = [int(x, 16) for x in v[1:]]
            rows.append((nums[0:4], nums[4:6], nums[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,want", _kat_rows())
def test_philox_known_answers(ctr, key, want):
    got = philox.philox4x32_10(np.array(ctr, dtype=np.uint32), key)
    assert [int(x) for x in got] == want


def test_uniform_end_points_exact():
    u = philox.uniforms(np.array([0, 511, 512, 0xFFFFFFFF], dtype=np.uint32))
    assert u[0] == 2.0 ** -24
    assert u[1] == 2.0 ** -24          # the low 9 bits are dropped
    assert u[2] == 3 * 2.0 ** -24
    assert u[3] == 1.0 - 2.0 ** -24
    assert np.all(u.astype(np.float32).astype(np.float64) == u)   # exact in fp32


def test_box_muller_special_values():
    # U0 = e^-1/2 gives radius 1; U1 = 0 -> angle 0, U1 = 1/4 -> angle pi/2.
    u = np.array([[np.exp(-0.5), 0.0, np.exp(-2.0), 0.25]])
    z = philox.box_muller(u)[0]
    assert z[0] == pytest.approx(1.0, abs=1e-15)
    assert z[1] == pytest.approx(0.0, abs=1e-15)
    assert z[2] == pytest.approx(0.0, abs=1e-15)
    assert z[3] == pytest.approx(2.0, abs=1e-15)


def test_value_noise_is_standard_normal():
    z = philox.value_noise(2, 0, 3, 8, np.arange(4096), 128).astype(np.float64).ravel()
    n = z.size
    assert abs(z.mean()) < 5.0 / np.sqrt(n)
    assert abs(z.var() - 1.0) < 6.0 * np.sqrt(2.0 / n)
    assert stats.kstest(z, "norm").pvalue > 1e-4
    # fourth moment of a standard normal is 3
    assert abs(np.mean(z ** 4) - 3.0) < 0.05


def test_value_noise_streams_are_distinct():
    base = philox.value_noise(2, 0, 0, 4, np.arange(256), 64)
    for other in (philox.value_noise(2, 1, 0, 4, np.arange(256), 64),   # another sequence
                  philox.value_noise(2, 0, 1, 4, np.arange(256), 64),   # another layer
                  philox.value_noise(3, 0, 0, 4, np.arange(256), 64)):  # another seed
        c = np.corrcoef(base.ravel(), other.ravel())[0, 1]
        assert abs(c) < 0.02
    # heads and positions differ too, and a position's draw does not depend on the others
    assert not np.array_equal(base[:, 0], base[:, 1])
    sub = philox.value_noise(2, 0, 0, 4, np.arange(100, 110), 64)
    assert np.array_equal(sub, base[100:110])
