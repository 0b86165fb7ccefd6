"""Pins for the oracle's noise generator (Philox4x32-10 + Box-Muller).

The known-answer vectors come from the generator's publication (file
tests/golden/philox4x32_10_kat.txt); the Gaussian law N(0, sigma^2 I) of the
noise is the paper's (Assumption 5), checked by moments and a KS test.
"""
import os

import numpy as np
import pytest
from scipy import stats

from oracle import philox as P
from conftest import GOLDEN


def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append([int(x, 16) for x in line.split()])
    return rows


@pytest.mark.parametrize("v", _kat())
def test_philox_known_answers(v):
    out = P.philox4x32_10(*v[:6])
    assert [int(o) for o in out] == v[6:]


def test_philox_vectorised_equals_scalar():
    rng = np.random.default_rng(5)
    c = rng.integers(0, 2**32, size=(6, 64), dtype=np.uint64)
    vec = P.philox4x32_10(*c)
    for j in range(64):
        sc = P.philox4x32_10(*(int(c[i, j]) for i in range(6)))
        assert [int(vec[i][j]) for i in range(4)] == [int(x) for x in sc]


def test_uniform_mapping_endpoints():
    u = P.word_to_uniform(np.array([0, 0xFF, 0x100, 0xFFFFFFFF], dtype=np.uint32))
    assert u[0] == 2.0 ** -24 and u[1] == 2.0 ** -24
    assert u[2] == 2.0 * 2.0 ** -24
    assert u[3] == 1.0
    # every value is exactly representable in float32
    assert np.all(u.astype(np.float32).astype(np.float64) == u)


def test_box_muller_special_points():
    ua = np.exp(-0.5)            # radius sqrt(-2 ln ua) = 1
    n0, n1 = P.box_muller(np.array([ua, ua, ua]), np.array([1.0, 0.25, 0.5]))
    np.testing.assert_allclose(n0, [1.0, 0.0, -1.0], atol=1e-15)
    np.testing.assert_allclose(n1, [0.0, 1.0, 0.0], atol=1e-15)


def test_gaussian_moments_and_law():
    # 1,048,576 draws from 2048 rows x 512 columns of one message
    xi = P.gaussian(0x5EED0005, 7, np.arange(2048), 512, P.TAG_EMB).ravel()
    n = xi.size
    se_mean = 1.0 / np.sqrt(n)
    se_var = np.sqrt(2.0 / n)
    assert abs(xi.mean()) < 5 * se_mean
    assert abs(xi.var() - 1.0) < 5 * se_var
    assert stats.kstest(xi[:200000], "norm").pvalue > 1e-3
    # the two outputs of one Box-Muller pair are uncorrelated
    a = P.gaussian(1, 0, np.arange(4096), 4, P.TAG_GRAD)
    assert abs(np.corrcoef(a[:, 0], a[:, 1])[0, 1]) < 5 / np.sqrt(4096)


def test_counter_layout():
    """Columns 4q..4q+3 of a row come from one Philox call with counter
    (step, row, q, tag); the tag and the step separate messages."""
    seed, step, row = 0x123456789, 11, 4242
    xi = P.gaussian(seed, step, np.array([row]), 8, P.TAG_EMB)[0]
    for q in range(2):
        w = P.philox4x32_10(step, row, q, P.TAG_EMB, seed & 0xFFFFFFFF, seed >> 32)
        ua, ub = P.word_to_uniform(w[0]), P.word_to_uniform(w[1])
        uc, ud = P.word_to_uniform(w[2]), P.word_to_uniform(w[3])
        a0, a1 = P.box_muller(ua, ub)
        b0, b1 = P.box_muller(uc, ud)
        np.testing.assert_array_equal(xi[4 * q:4 * q + 4], [a0, a1, b0, b1])
    other = P.gaussian(seed, step, np.array([row]), 8, P.TAG_GRAD)[0]
    later = P.gaussian(seed, step + 1, np.array([row]), 8, P.TAG_EMB)[0]
    assert not np.any(other == xi) and not np.any(later == xi)
