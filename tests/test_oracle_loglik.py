"""Pins for the oracle's log-likelihood over draws (Section 3.2): the
textbook Bernoulli form written differently (y log sigma + (1 - y) log(1 -
sigma) with scipy's log-expit), closed forms for X = 0 and equal draws, the
library logsumexp, and the relation to the potential."""
import numpy as np
from scipy import special

import workloads


def test_matches_textbook_bernoulli(orc):
    X, y, _ = workloads.make_logistic(300, 7, w_scale=1.5, key=[80, 1])
    rng = np.random.default_rng(2)
    W = rng.normal(0.0, 1.2, size=(9, 7))
    ll, pm = orc.log_likelihood(X, y, W)
    eta = X @ W.T                                           # [N, S]
    yy = y[:, None].astype(np.float64)
    ref = (yy * special.log_expit(eta) + (1 - yy) * special.log_expit(-eta)).sum(axis=0)
    np.testing.assert_allclose(ll, ref, rtol=1e-12)
    np.testing.assert_allclose(pm, special.expit(eta).mean(axis=1), rtol=1e-12)


def test_closed_forms(orc):
    # X = 0: every row has probability 1/2 whatever the draw
    X = np.zeros((50, 3))
    y = (np.arange(50) % 3 == 0).astype(np.uint8)
    ll, pm = orc.log_likelihood(X, y, np.random.default_rng(3).normal(size=(4, 3)))
    np.testing.assert_allclose(ll, -50 * np.log(2.0), rtol=1e-14)
    assert np.all(pm == 0.5)
    # one row x = [1], y = 1, w = log 3: sigma = 3/4
    ll, pm = orc.log_likelihood(np.ones((1, 1)), np.ones(1, np.uint8), np.array([[np.log(3.0)]]))
    np.testing.assert_allclose(ll, [np.log(0.75)], rtol=1e-15)
    np.testing.assert_allclose(pm, [0.75], rtol=1e-15)


def test_expected_log_likelihood(orc):
    rng = np.random.default_rng(4)
    ll = rng.normal(-3000.0, 40.0, size=500)
    np.testing.assert_allclose(orc.expected_log_likelihood(ll),
                               special.logsumexp(ll) - np.log(ll.size), rtol=1e-14)
    # equal draws: the average of equal likelihoods is that likelihood
    assert orc.expected_log_likelihood(np.full(7, -12.5)) == -12.5


def test_relation_to_potential(orc):
    X, y, _ = workloads.make_logistic(200, 5, w_scale=1.0, key=[80, 2])
    W = np.random.default_rng(5).normal(size=(3, 5))
    ll, _ = orc.log_likelihood(X, y, W)
    s = 1.7
    for k in range(3):
        U, _ = orc.logistic_potential_grad(X, y, W[k], prior_scale=s)
        prior = 0.5 * np.sum(W[k] ** 2) / s**2 + 5 * (np.log(s) + 0.5 * np.log(2 * np.pi))
        np.testing.assert_allclose(-ll[k], U - prior, rtol=1e-12)
