"""GPU parity of the log-likelihood over draws (nuts_data_log_likelihood)
against the oracle.

Bars.  fp32 data (matrix-core path): products, row terms and the per-tile
sums of sigmoid run in fp32, so every row term carries a relative error of
a few fp32 ulps; the sums are fp64.  ll[s] is a sum of N non-negative terms,
so its error is within 1e-5 of its magnitude (the batched potential's bar);
the expected log-likelihood is 1-Lipschitz in the largest ll error; the
predictive means are averages of probabilities in [0, 1] and sit within
1e-5 absolute.  fp64 data (streaming path): ll comes from the fp64
potential with the prior taken off, within 1e-10 of |U| + prior.
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


def _draws(S, D, key, scale=0.4):
    return np.random.default_rng(key).normal(0.0, scale, size=(S, D))


@pytest.mark.parametrize("N,D,S", [
    (1, 3, 1),            # one row, one draw
    (100, 9, 5),          # ragged stage, chunk padding
    (1000, 20, 130),      # tail columns, two tiles (the second nearly empty)
    (5000, 55, 256),      # the covtype width
    (3001, 129, 300),     # widest matrix-core shape, three tiles
])
def test_fp32_matches_oracle(sampler, orc, N, D, S):
    X, y, _ = workloads.make_logistic(N, D, w_scale=0.5, key=[90, N * 1000 + D], dtype="f32")
    W = _draws(S, D, [91, S])
    say("loglik fp32", N, D, S)
    d = sampler.data(X, y)
    ll, elpd, pm = d.log_likelihood(W, pred_mean=True)
    ref_ll, ref_pm = orc.log_likelihood(X.astype(np.float64), y, W)
    np.testing.assert_allclose(ll, ref_ll, rtol=1e-5)
    err = np.max(np.abs(ll - ref_ll))
    assert abs(elpd - orc.expected_log_likelihood(ref_ll)) <= err + 1e-9 * abs(elpd)
    np.testing.assert_allclose(pm, ref_pm, atol=1e-5)
    d.free()


@pytest.mark.parametrize("N,D,S", [(1, 1, 1), (777, 11, 40), (3000, 257, 7)])
def test_fp64_matches_oracle(sampler, orc, N, D, S):
    X, y, _ = workloads.make_logistic(N, D, w_scale=0.5, key=[92, N * 1000 + D])
    W = _draws(S, D, [93, S])
    say("loglik fp64", N, D, S)
    d = sampler.data(X, y)
    ll, elpd, pm = d.log_likelihood(W)
    assert pm is None
    ref_ll, _ = orc.log_likelihood(X, y, W)
    bound = 1e-10 * (np.abs(ref_ll) + 0.5 * np.sum(W**2, axis=1) + D)
    assert np.all(np.abs(ll - ref_ll) <= bound), np.max(np.abs(ll - ref_ll) / bound)
    np.testing.assert_allclose(elpd, orc.expected_log_likelihood(ref_ll), rtol=1e-10)
    d.free()


def test_full_size_sampled_draws(sampler, orc):
    # the covtype-shaped fp32 set with 500 draws (four tiles), as the timed
    # call runs it; four draws checked against the oracle one by one
    wl = workloads.WORKLOADS["covtype_n581012_d55_f32"]
    X, y, w_true = workloads.make_logistic(wl.N, wl.D, w_scale=wl.w_scale, key=wl.data_seed,
                                           dtype=wl.dtype)
    W = w_true[None, :] + _draws(500, wl.D, [94, 1], scale=0.003)
    say("loglik full size", wl.N, wl.D, 500)
    d = sampler.data(X, y)
    ll, elpd, pm = d.log_likelihood(W, pred_mean=True)
    idx = [0, 127, 128, 499]
    ref_ll, ref_pm = orc.log_likelihood(X.astype(np.float64), y, W[idx])
    np.testing.assert_allclose(ll[idx], ref_ll, rtol=1e-5)
    # the predictive mean of a few rows, from all 500 draws
    rows = [0, 1, 65, wl.N - 1]
    _, pm_rows = orc.log_likelihood(X[rows].astype(np.float64), y[rows], W)
    np.testing.assert_allclose(pm[rows], pm_rows, atol=1e-5)
    assert np.all((pm >= 0) & (pm <= 1))
    d.free()


def test_rejects(sampler):
    import paper_1912_11554_amd as nuts
    X64, y64, _ = workloads.make_logistic(50, 4, w_scale=0.5, key=[95, 1])
    d = sampler.data(X64, y64)
    with pytest.raises(nuts.NutsError) as e:
        d.log_likelihood(np.zeros((2, 4)), pred_mean=True)  # fp64 data: no predictive mean
    assert e.value.code == nuts.NUTS_EUNSUPPORTED
    d.free()
    Xc, yc = np.zeros((2, 30, 3)), np.zeros((2, 30), np.uint8)
    dc = sampler.data(Xc, yc, per_chain=True)
    with pytest.raises(nuts.NutsError) as e:
        dc.log_likelihood(np.zeros((1, 3)))
    assert e.value.code == nuts.NUTS_EINVAL
    dc.free()
