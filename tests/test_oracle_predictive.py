"""Pins for the oracle's posterior predictive samples (reading R23): at a
draw with x . w = 0 every probability is 1/2 and y is the complement of the
top bit of the row's Philox word, taken from numpy's independent Philox; at
varied probabilities the frequencies over 4000 independently keyed draws
match sigmoid(x . w) within binomial error; rows sharing a Philox block are
uncorrelated; the returned probabilities are the logistic of x . w."""
import numpy as np
from scipy.special import expit

from tests.test_oracle_rng import _numpy_block


def test_half_probability_is_the_top_bit(orc):
    X = np.random.default_rng(1).normal(size=(11, 3))
    W = np.zeros((3, 3))
    seed = 77
    y, p = orc.posterior_predictive(X, W, seed)
    assert np.all(p == 0.5)
    for s in range(3):
        for i in range(11):
            word = int(_numpy_block([0, 7 << 32, i // 4, 0], [seed, s])[i % 4])
            # u < 1/2 iff the top bit of the 53-bit uniform is clear
            assert y[s, i] == (1 if (word >> 63) == 0 else 0), (s, i)


def test_frequencies_match_probabilities(orc):
    rng = np.random.default_rng(2)
    N, D, S = 40, 4, 4000
    X = rng.normal(size=(N, D))
    w = rng.normal(size=D)
    W = np.repeat(w[None, :], S, axis=0)
    y, p = orc.posterior_predictive(X, W, 5)
    pr = expit(X @ w)
    np.testing.assert_allclose(p[0], pr, rtol=1e-12, atol=1e-15)
    freq = y.mean(axis=0)
    sd = np.sqrt(pr * (1 - pr) / S) + 1e-12
    assert np.all(np.abs(freq - pr) < 4.5 * sd + 1.0 / S)
    assert pr.min() < 0.1 and pr.max() > 0.9
    # rows 0 and 1 use words of the same block: no correlation
    c = np.corrcoef(y[:, 0].astype(float), y[:, 1].astype(float))[0, 1]
    assert abs(c) < 4.5 / np.sqrt(S)


def test_keys_differ_by_seed_and_draw(orc):
    X = np.ones((64, 1))
    W = np.zeros((2, 1))
    a, _ = orc.posterior_predictive(X, W, 1)
    b, _ = orc.posterior_predictive(X, W, 2)
    assert not np.array_equal(a[0], a[1])
    assert not np.array_equal(a, b)
