"""GPU parity of the posterior predictive samples
(nuts_data_posterior_predictive) against the oracle.

Both sides draw the same keyed uniform u for each (draw, row) and output
y = [u < sigmoid(x . w)]; the device's probability comes from fp32
products and an fp32 sigmoid, the oracle's from fp64.  With |eta| error at
most 1e-6 (1 + sum_j |x_ij w_j|) (fp32 products of fp32 X and W rounded to
fp32) and the sigmoid's slope at most 1/4, the two probabilities differ by
less than 5e-7 (1 + sum_j |x_ij w_j|) + 1e-6: a sample may differ only
where u lies that close to the oracle's probability, and everywhere else it
must be identical.
"""
import numpy as np
import pytest

import workloads
from tests.gpu_common import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sampler():
    import paper_1912_11554_amd as nuts
    return nuts.Sampler(0)


def _check(y, X, W, seed, orc, first_draw=0):
    X64 = np.asarray(X, dtype=np.float64)
    yr, p, u = orc.posterior_predictive(X64, W, seed, uniforms=True, first_draw=first_draw)
    mag = np.abs(X64) @ np.abs(W).T  # [N, S]
    bound = (5e-7 * (1.0 + mag) + 1e-6).T
    diff = y != yr
    near = np.abs(u - p) <= bound
    assert not np.any(diff & ~near), np.argwhere(diff & ~near)[:5]
    return int(diff.sum())


@pytest.mark.parametrize("N,D,S", [(1, 3, 1), (100, 9, 5), (1000, 20, 130), (5000, 55, 256),
                                   (3001, 129, 300)])
def test_matches_oracle(sampler, orc, N, D, S):
    X, y, _ = workloads.make_logistic(N, D, w_scale=0.5, key=[96, N * 1000 + D], dtype="f32")
    W = np.random.default_rng([97, S]).normal(0.0, 0.6, size=(S, D))
    say("predictive", N, D, S)
    d = sampler.data(X, y)
    yy = d.posterior_predictive(W, seed=123)
    assert yy.shape == (S, N) and set(np.unique(yy)) <= {0, 1}
    _check(yy, X, W, 123, orc)
    # another seed gives other samples
    if N * S >= 1000:
        assert not np.array_equal(yy, d.posterior_predictive(W, seed=124))
    d.free()


def test_full_size_sampled_draws(sampler, orc):
    # the covtype-shaped fp32 set with 500 draws (four tiles of 128), five
    # draws checked against the oracle over every row
    wl = workloads.WORKLOADS["covtype_n581012_d55_f32"]
    X, y, w_true = workloads.make_logistic(wl.N, wl.D, w_scale=wl.w_scale, key=wl.data_seed,
                                           dtype=wl.dtype)
    W = w_true[None, :] + np.random.default_rng([98, 1]).normal(0.0, 0.003, size=(500, wl.D))
    say("predictive full size", wl.N, wl.D, 500)
    d = sampler.data(X, y)
    yy = d.posterior_predictive(W, seed=9)
    for s in (0, 127, 128, 255, 499):
        _check(yy[s:s + 1], X, W[s:s + 1], 9, orc, first_draw=s)
    # the sample mean over draws tracks the predictive mean of the same draws
    _, _, pm = d.log_likelihood(W, pred_mean=True)
    assert np.abs(yy.mean(axis=0) - pm).max() < 6.0 * np.sqrt(0.25 / 500) + 1e-3
    d.free()


def test_rejects(sampler):
    import paper_1912_11554_amd as nuts
    X64, y64, _ = workloads.make_logistic(50, 4, w_scale=0.5, key=[99, 1])
    d = sampler.data(X64, y64)
    with pytest.raises(nuts.NutsError) as e:
        d.posterior_predictive(np.zeros((2, 4)))
    assert e.value.code == nuts.NUTS_EUNSUPPORTED
    d.free()
