"""Pins for the oracle's potential U and gradient of the logistic log-joint
(Appendix B model: m ~ N(0, 1), b ~ N(0, 1), y ~ Bernoulli(logits = x.m + b),
intercept folded in as a ones column).

Independent references: the closed form at w = 0, scipy's Bernoulli and
Normal log densities, torch autograd through torch.distributions (fp64, CPU),
central finite differences of U itself, and the special cases that reduce
to the Gaussian prior.
"""
import numpy as np
import pytest
import torch
from scipy import special, stats

import workloads


def _data(N, D, seed, w_scale=1.0):
    X, y, w = workloads.make_logistic(N, D, w_scale=w_scale, key=seed)
    return X, y, w


def test_closed_form_at_zero(orc):
    X, y, _ = _data(300, 7, 1)
    for s in (1.0, 0.5, 3.0):
        U, g = orc.logistic_potential_grad(X, y, np.zeros(7), prior_scale=s)
        N, D = X.shape
        assert U == pytest.approx(N * np.log(2.0) + D * (np.log(s) + 0.5 * np.log(2 * np.pi)),
                                  rel=1e-14)
        np.testing.assert_allclose(g, -X.T @ (y - 0.5), rtol=1e-13, atol=1e-12)


@pytest.mark.parametrize("s", [1.0, 0.7])
def test_matches_scipy_log_densities(orc, s):
    X, y, w_true = _data(500, 9, 2)
    rng = np.random.default_rng(0)
    for _ in range(5):
        w = w_true + 0.3 * rng.normal(size=9)
        U, _ = orc.logistic_potential_grad(X, y, w, prior_scale=s)
        p = special.expit(X @ w)
        ref = -stats.bernoulli.logpmf(y, p).sum() - stats.norm.logpdf(w, 0.0, s).sum()
        assert U == pytest.approx(ref, rel=1e-11)


def test_matches_torch_autograd(orc):
    X, y, w_true = _data(700, 12, 3, w_scale=2.0)
    rng = np.random.default_rng(1)
    for scale in (0.0, 1.0, 5.0):
        w = w_true + scale * rng.normal(size=12)
        Xt = torch.tensor(X, dtype=torch.float64)
        wt = torch.tensor(w, dtype=torch.float64, requires_grad=True)
        yt = torch.tensor(y, dtype=torch.float64)
        lp = torch.distributions.Bernoulli(logits=Xt @ wt).log_prob(yt).sum()
        lp = lp + torch.distributions.Normal(0.0, 1.0).log_prob(wt).sum()
        (-lp).backward()
        U, g = orc.logistic_potential_grad(X, y, w)
        assert U == pytest.approx(-lp.item(), rel=1e-12)
        np.testing.assert_allclose(g, wt.grad.numpy(), rtol=1e-11,
                                   atol=1e-11 * np.abs(wt.grad.numpy()).max())


def test_gradient_finite_differences(orc):
    X, y, w_true = _data(400, 6, 4)
    w = w_true + 0.1
    U0, g = orc.logistic_potential_grad(X, y, w)
    h = 1e-5
    fd = np.zeros(6)
    for j in range(6):
        e = np.zeros(6)
        e[j] = h
        up = orc.logistic_potential_grad(X, y, w + e)[0]
        um = orc.logistic_potential_grad(X, y, w - e)[0]
        up2 = orc.logistic_potential_grad(X, y, w + 2 * e)[0]
        um2 = orc.logistic_potential_grad(X, y, w - 2 * e)[0]
        fd[j] = (-up2 + 8 * up - 8 * um + um2) / (12 * h)
    np.testing.assert_allclose(fd, g, rtol=1e-7, atol=1e-7 * np.abs(g).max())


def test_saturating_logits(orc):
    # |eta| = 50: a correct label costs ~exp(-50), a wrong one ~50; the
    # residual is exactly representable as -exp(-50) or +1 (up to rounding)
    X = np.array([[50.0], [-50.0], [50.0], [-50.0]])
    y = np.array([1, 0, 0, 1], dtype=np.uint8)
    U, g = orc.logistic_potential_grad(X, y, np.array([1.0]), prior_scale=1e6)
    prior = 0.5 / 1e12 + np.log(1e6) + 0.5 * np.log(2 * np.pi)
    want = 2 * np.log1p(np.exp(-50.0)) + 2 * (50.0 + np.log1p(np.exp(-50.0)))
    assert U - prior == pytest.approx(want, rel=1e-14)
    # rows 0,1 correct: r x = -e^-50 * 50 each; rows 2,3 wrong: +50 each
    r_small = 50.0 * np.exp(-50.0) / (1 + np.exp(-50.0))
    assert g[0] == pytest.approx(-2 * r_small + 2 * 50.0 / (1 + np.exp(-50.0)) + 1e-12,
                                 rel=1e-14)
    # every row term -log p(y_i | x_i, w) is >= 0
    X, y, _ = _data(200, 5, 5)
    w = np.ones(5) * 3
    prior_U = -stats.norm.logpdf(w, 0.0, 1.0).sum()
    row_terms = [orc.logistic_potential_grad(X[i:i + 1], y[i:i + 1], w)[0] - prior_U
                 for i in range(50)]
    assert min(row_terms) >= 0.0


def test_no_data_reduces_to_prior(orc):
    rng = np.random.default_rng(3)
    w = rng.normal(size=5)
    for s in (1.0, 2.5):
        prior_U = -stats.norm.logpdf(w, 0.0, s).sum()
        # X = 0: every row costs exactly ln 2 and contributes no gradient
        U, g = orc.logistic_potential_grad(np.zeros((10, 5)), np.ones(10, np.uint8), w, s)
        assert U == pytest.approx(prior_U + 10 * np.log(2.0), rel=1e-14)
        np.testing.assert_allclose(g, w / s**2, rtol=1e-14)
        # N = 0
        U, g = orc.logistic_potential_grad(np.zeros((0, 5)), np.zeros(0, np.uint8), w, s)
        assert U == pytest.approx(prior_U, rel=1e-14)
        np.testing.assert_allclose(g, w / s**2, rtol=1e-14)


def test_f32_variant_equals_promoted_f64(orc):
    X, y, w = _data(333, 7, 6)
    Xf = X.astype(np.float32)
    U1, g1 = orc.logistic_potential_grad_f32(Xf, y, w)
    U2, g2 = orc.logistic_potential_grad(Xf.astype(np.float64), y, w)
    assert U1 == U2
    assert np.array_equal(g1, g2)


def test_lingauss_target(orc):
    X, yv = workloads.make_lingauss(50, 4, key=7, noise_scale=0.5)
    rng = np.random.default_rng(4)
    w1, w2 = rng.normal(size=4), rng.normal(size=4)
    U1, g1 = orc.lingauss_potential_grad(X, yv, w1, 2.0, 0.5)
    U2, _ = orc.lingauss_potential_grad(X, yv, w2, 2.0, 0.5)
    lp = lambda w: (stats.norm.logpdf(yv, X @ w, 0.5).sum()
                    + stats.norm.logpdf(w, 0, 2.0).sum())
    assert U1 - U2 == pytest.approx(-(lp(w1) - lp(w2)), rel=1e-10)
    # gradient: torch autograd of the same log density
    wt = torch.tensor(w1, requires_grad=True)
    Xt = torch.tensor(X)
    l = (torch.distributions.Normal(Xt @ wt, 0.5).log_prob(torch.tensor(yv)).sum()
         + torch.distributions.Normal(0.0, 2.0).log_prob(wt).sum())
    (-l).backward()
    np.testing.assert_allclose(g1, wt.grad.numpy(), rtol=1e-11)
