"""Pins for the ESS estimator against closed forms: an AR(1) series with
coefficient phi has integrated autocorrelation time (1 + phi) / (1 - phi)."""
import numpy as np
import pytest

from oracle.ess import ess, mcse_mean


def _ar1(phi, n, rng, C=1):
    e = rng.normal(size=(C, n))
    x = np.zeros((C, n))
    x[:, 0] = e[:, 0]
    a = np.sqrt(1 - phi * phi)
    for t in range(1, n):
        x[:, t] = phi * x[:, t - 1] + a * e[:, t]
    return x


@pytest.mark.parametrize("phi", [0.0, 0.5, 0.9, -0.4])
def test_ar1_closed_form(phi):
    rng = np.random.default_rng(int(abs(phi) * 100))
    n = 200000
    x = _ar1(phi, n, rng)[0]
    want = n * (1 - phi) / (1 + phi)
    assert ess(x) == pytest.approx(want, rel=0.1)


def test_multi_chain():
    rng = np.random.default_rng(7)
    x = _ar1(0.8, 20000, rng, C=4)
    want = 4 * 20000 * 0.2 / 1.8
    assert ess(x) == pytest.approx(want, rel=0.1)
    # chains stuck in different places: between-chain variance lowers the ESS
    shifted = x + np.arange(4)[:, None] * 3.0
    assert ess(shifted) < 0.1 * want


def test_mcse_of_iid_mean():
    rng = np.random.default_rng(3)
    x = rng.normal(size=(50000, 2)) * np.array([1.0, 3.0])
    np.testing.assert_allclose(mcse_mean(x), np.array([1.0, 3.0]) / np.sqrt(50000), rtol=0.1)
