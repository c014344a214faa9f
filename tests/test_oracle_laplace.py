"""Pins for the oracle's normal approximation of the logistic posterior
(Appendix B model): the MAP by Newton's method, the Laplace covariance and the
skewness-corrected posterior mean.  The GPU sampler's long fp32 runs are
checked against these where no oracle sampler can run long enough.

Independent references: the gradient of U (itself pinned in
test_oracle_target.py) vanishing at the MAP; a central finite-difference
Hessian of that gradient; one- and two-dimensional posteriors integrated
numerically (scipy quadrature, a dense grid), whose exact mean the corrected
mean must approach at order 1/N^2 while the mode is off at order 1/N.
"""
import numpy as np
import pytest
from scipy import integrate, optimize, special

import workloads


@pytest.mark.parametrize("N,D,s,ws", [(300, 4, 1.0, 1.0), (2000, 9, 0.5, 1.0), (5000, 17, 2.0, 0.3)])
def test_gradient_vanishes_at_map(orc, N, D, s, ws):
    X, y, _ = workloads.make_logistic(N, D, w_scale=ws, key=[81, 100 * N + D])
    r = orc.logistic_laplace(X, y, s)
    _, g = orc.logistic_potential_grad(X, y, r["w_map"], s)
    # each gradient component is a sum of terms |r_i x_ij| <= |x_ij|
    scale = np.abs(X).sum(axis=0) + np.abs(r["w_map"]) / s**2 + 1.0
    assert np.all(np.abs(g) <= 1e-10 * scale), np.abs(g) / scale
    assert 2 <= r["newton_steps"] <= 30


def test_fp32_rows_equal_promoted(orc):
    X, y, _ = workloads.make_logistic(700, 6, w_scale=1.0, key=82, dtype="f32")
    a = orc.logistic_laplace(X, y)
    b = orc.logistic_laplace(X.astype(np.float64), y)
    for k in ("w_map", "cov", "mean"):
        assert np.array_equal(a[k], b[k]), k


def test_covariance_is_inverse_fd_hessian(orc):
    N, D = 1500, 6
    X, y, _ = workloads.make_logistic(N, D, w_scale=1.0, key=83)
    r = orc.logistic_laplace(X, y, 1.0)
    w = r["w_map"]
    h = 1e-5
    H = np.zeros((D, D))
    for j in range(D):
        e = np.zeros(D)
        e[j] = h
        gp = orc.logistic_potential_grad(X, y, w + e)[1]
        gm = orc.logistic_potential_grad(X, y, w - e)[1]
        H[:, j] = (gp - gm) / (2 * h)
    H = 0.5 * (H + H.T)
    np.testing.assert_allclose(r["cov"], np.linalg.inv(H), rtol=1e-6,
                               atol=1e-6 * np.abs(r["cov"]).max())
    # symmetric positive definite
    np.testing.assert_allclose(r["cov"], r["cov"].T, rtol=0, atol=1e-13 * np.abs(r["cov"]).max())
    assert np.linalg.eigvalsh(r["cov"]).min() > 0


def _intercept_only_exact(N, k, s):
    """Mode, mean and variance of p(b) ~ sigmoid(b)^k sigmoid(-b)^(N-k) N(b; 0, s^2)
    by root finding and adaptive quadrature."""
    lp = lambda b: k * special.log_expit(b) + (N - k) * special.log_expit(-b) - 0.5 * b * b / s**2
    dlp = lambda b: k * special.expit(-b) - (N - k) * special.expit(b) - b / s**2
    m = optimize.brentq(dlp, -30.0, 30.0, xtol=1e-15, rtol=1e-15)
    c = lp(m)
    kw = dict(epsabs=0.0, epsrel=1e-13, limit=400)
    Z = integrate.quad(lambda b: np.exp(lp(b) - c), m - 30, m + 30, **kw)[0]
    M = integrate.quad(lambda b: b * np.exp(lp(b) - c), m - 30, m + 30, **kw)[0] / Z
    V = integrate.quad(lambda b: (b - M) ** 2 * np.exp(lp(b) - c), m - 30, m + 30, **kw)[0] / Z
    curv = N * special.expit(m) * special.expit(-m) + 1.0 / s**2
    return m, M, V, curv


def test_intercept_only_against_quadrature(orc):
    # one column of ones: the posterior of the intercept alone, in closed
    # form up to one-dimensional integrals
    errs = []
    for N in (50, 200, 800):
        k = (4 * N) // 5
        X = np.ones((N, 1))
        y = np.zeros(N, np.uint8)
        y[:k] = 1
        r = orc.logistic_laplace(X, y, 1.0)
        m, M, V, curv = _intercept_only_exact(N, k, 1.0)
        assert r["w_map"][0] == pytest.approx(m, abs=1e-12)
        assert r["cov"][0, 0] == pytest.approx(1.0 / curv, rel=1e-12)
        mode_err = abs(r["w_map"][0] - M)
        corr_err = abs(r["mean"][0] - M)
        assert corr_err < 0.02 * mode_err, (N, corr_err, mode_err)
        errs.append((mode_err, corr_err))
    # the mode is off at order 1/N, the corrected mean at order 1/N^2
    assert 2.5 < errs[1][0] / errs[2][0] < 5.5
    assert errs[1][1] / errs[2][1] > 8.0


@pytest.mark.parametrize("N", [40, 160])
def test_two_dimensional_posterior_on_a_grid(orc, N):
    # a feature and the intercept: the posterior mean and covariance by a
    # dense grid over +-12 Laplace standard deviations
    X, y, _ = workloads.make_logistic(N, 2, w_scale=1.0, key=[84, N])
    r = orc.logistic_laplace(X, y, 1.0)
    sd = np.sqrt(np.diag(r["cov"]))
    g0 = np.linspace(r["w_map"][0] - 12 * sd[0], r["w_map"][0] + 12 * sd[0], 1201)
    g1 = np.linspace(r["w_map"][1] - 12 * sd[1], r["w_map"][1] + 12 * sd[1], 1201)
    A, B = np.meshgrid(g0, g1, indexing="ij")
    lp = -0.5 * (A**2 + B**2)
    for i in range(N):
        eta = X[i, 0] * A + X[i, 1] * B
        lp += special.log_expit(eta) if y[i] else special.log_expit(-eta)
    p = np.exp(lp - lp.max())
    p /= p.sum()
    M = np.array([(A * p).sum(), (B * p).sum()])
    C01 = ((A - M[0]) * (B - M[1]) * p).sum()
    C = np.array([[((A - M[0]) ** 2 * p).sum(), C01], [C01, ((B - M[1]) ** 2 * p).sum()]])
    mode_err = np.abs(r["w_map"] - M) / sd
    corr_err = np.abs(r["mean"] - M) / sd
    assert mode_err.max() > 0.02  # the skewness is visible at this N
    assert np.all(corr_err < 0.1 * mode_err.max()), (corr_err, mode_err)
    # the Laplace covariance is off at order 1/N
    assert np.abs((r["cov"] - C) / np.outer(sd, sd)).max() < 10.0 / N
