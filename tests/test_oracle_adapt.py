"""Pins for the oracle's warmup adaptation (reading R19): the window
schedule of the windowed diagonal-mass scheme, the dual-averaging recursion
of Hoffman & Gelman (2014, Section 3.2) against its closed form, their
step-size heuristic (Alg. 4) against the closed-form leapfrog of a Gaussian,
and the statistical consequences: the adapted step size reaches the target
acceptance, and the adapted inverse mass follows the posterior variances
while sampling stays exact."""
import numpy as np
import pytest

import workloads
from oracle.ess import ess_columns

LN2 = np.log(2.0)


def test_mass_windows_published_default(orc):
    # The Stan reference manual's example for 1000 warmup iterations: an
    # initial buffer of 75, slow windows of 25, 50, 100, 200 and a last one
    # stretched to 500 iterations, then a terminal buffer of 50.
    assert orc.mass_windows(1000) == [(75, 100), (100, 150), (150, 250), (250, 450), (450, 950)]
    assert orc.mass_windows(19) == []


@pytest.mark.parametrize("W", [20, 37, 100, 149, 150, 151, 200, 300, 600, 1000, 2000, 5000])
def test_mass_windows_structure(orc, W):
    win = orc.mass_windows(W)
    if W >= 150:
        init, term, base = 75, 50, 25
    else:
        init, term = int(0.15 * W), int(0.1 * W)
        base = W - init - term
    assert win[0][0] == init and win[-1][1] == W - term
    for (a, b), (c, d) in zip(win, win[1:]):
        assert b == c                                   # contiguous
    sizes = [b - a for a, b in win]
    assert sizes[0] == base or len(win) == 1
    for k in range(1, len(sizes) - 1):
        assert sizes[k] == 2 * sizes[k - 1]             # doubling
    if len(sizes) > 1:
        # the last window took over the remainder because a doubled window
        # after it would not fit
        assert sizes[-1] >= 2 * sizes[-2]
        assert win[-1][0] + 2 * sizes[-2] + 4 * sizes[-2] > W - term


def test_dual_averaging_closed_form(orc):
    # With a constant accept statistic alpha the recursion
    #   Hbar_m = (1 - 1/(m + t0)) Hbar_{m-1} + (delta - alpha)/(m + t0),  Hbar_0 = 0
    # has the closed form Hbar_m = (delta - alpha) m / (m + t0) (induction:
    # (m + t0 - 1)/(m + t0) * (m - 1)/(m - 1 + t0) + 1/(m + t0) = m/(m + t0)),
    # so log eps_m = mu - sqrt(m)/gamma * (delta - alpha) m/(m + t0) with
    # mu = log(10 eps0), gamma = 0.05, t0 = 10.
    eps0, delta, t0, gamma = 0.37, 0.8, 10.0, 0.05
    m = np.arange(1, 301, dtype=np.float64)
    for alpha in (0.6, 0.95, 0.8):
        le, lb = orc.dual_averaging(eps0, delta, np.full(m.size, alpha))
        want = np.log(10 * eps0) - np.sqrt(m) / gamma * (delta - alpha) * m / (m + t0)
        np.testing.assert_allclose(le, want, rtol=1e-13, atol=1e-13)
        # the first average has weight 1 on the first iterate
        assert lb[0] == le[0]
        if alpha == delta:
            np.testing.assert_allclose(lb, np.log(10 * eps0), rtol=1e-15)
        # too low an acceptance shrinks the step, too high a one grows it
        assert np.all(le[1:] < le[0]) if alpha < delta else True
        assert np.all(le[1:] > le[0]) if alpha > delta else True
    # eps_bar is a running average: it lies between the smallest and the
    # largest iterate seen so far
    rng = np.random.default_rng(3)
    a = rng.uniform(0.3, 1.0, 200)
    le, lb = orc.dual_averaging(eps0, delta, a)
    for i in range(1, 200):
        assert le[: i + 1].min() - 1e-12 <= lb[i] <= le[: i + 1].max() + 1e-12


def _gauss_dH(q, p, eps, prec):
    """H(start) - H(after one leapfrog step) for U = prec q^2 / 2, unit mass:
    the leapfrog map is linear, [q'; p'] = A [q; p] with
    A = [[1 - e^2 w^2/2, e], [-e w^2 (1 - e^2 w^2/4), 1 - e^2 w^2/2]], w^2 = prec."""
    w2 = prec
    a11 = 1.0 - eps * eps * w2 / 2.0
    q1 = a11 * q + eps * p
    p1 = -eps * w2 * (1.0 - eps * eps * w2 / 4.0) * q + a11 * p
    return (0.5 * prec * q * q + 0.5 * p * p) - (0.5 * prec * q1 * q1 + 0.5 * p1 * p1)


@pytest.mark.parametrize("q0,eps0,seed", [(0.3, 1e-3, 1), (1.2, 0.01, 2), (-0.5, 40.0, 3),
                                          (0.0, 3.0, 4), (2.0, 0.5, 5), (-1.0, 1e-5, 6)])
def test_find_step_size_gaussian(orc, q0, eps0, seed):
    # one-dimensional Gaussian posterior: one observation yv = 0 with unit
    # noise through x = a, prior scale s; precision a^2 + 1/s^2
    a, s = 1.7, 3.0
    prec = a * a + 1.0 / (s * s)
    X = np.array([[a]])
    yv = np.array([0.0])
    eps, evals = orc.find_step_size(X, None, np.array([q0]), eps0, seed=seed, t=9,
                                    prior_scale=s, target=orc.TARGET_LINGAUSS, yv=yv,
                                    noise_scale=1.0)
    r = orc.normals(seed, 0, 9, 1, tag=5)[0]
    d0 = _gauss_dH(q0, r, eps0, prec)
    up = d0 > -LN2
    k = int(round(np.log2(eps / eps0)))
    assert eps == eps0 * 2.0**k and (k > 0 if up else k < 0)
    # every step size tried before the last kept (up) or lost (down) more
    # than half the density, the last one did not
    for i in range(abs(k)):
        e = eps0 * 2.0 ** (i if up else -i)
        assert (_gauss_dH(q0, r, e, prec) > -LN2) == up
    dk = _gauss_dH(q0, r, eps, prec)
    assert (dk > -LN2) != up or (not up and dk == -LN2)
    assert evals == 1 + abs(k) + 1  # the gradient at q0, then one leapfrog per trial


@pytest.mark.slow
@pytest.mark.parametrize("delta", [0.8, 0.95])
def test_adapted_step_reaches_target_acceptance(orc, delta):
    X, yv = workloads.make_lingauss(40, 4, key=77, noise_scale=0.7)
    res = [orc.nuts(X, None, step_size=1e-3, max_tree_depth=10, num_warmup=500, num_samples=600,
                    seed=11, chain=c, prior_scale=2.0, target=orc.TARGET_LINGAUSS, yv=yv,
                    noise_scale=0.7, adapt_step_size=True, target_accept=delta)
           for c in range(3)]
    acc = np.concatenate([r["stats"]["accept_prob"] for r in res])
    assert abs(acc.mean() - delta) < 0.06, acc.mean()
    eps = [r["step_size"] for r in res]
    assert all(e > 1e-3 * 4 for e in eps)  # moved well away from the start


@pytest.mark.slow
def test_higher_target_gives_smaller_step(orc):
    X, yv = workloads.make_lingauss(40, 4, key=77, noise_scale=0.7)
    kw = dict(step_size=0.05, max_tree_depth=10, num_warmup=500, num_samples=10, seed=12,
              prior_scale=2.0, target=orc.TARGET_LINGAUSS, yv=yv, noise_scale=0.7,
              adapt_step_size=True)
    lo = orc.nuts(X, None, target_accept=0.6, **kw)["step_size"]
    hi = orc.nuts(X, None, target_accept=0.95, **kw)["step_size"]
    assert hi < lo


@pytest.mark.slow
def test_windowed_mass_follows_posterior_variances(orc):
    # strongly anisotropic Gaussian posterior (sds 0.05, 1, 20): after the
    # windowed warmup the inverse mass (not normalised) is the posterior
    # variance, and the samples keep the right moments
    sds = np.array([0.05, 1.0, 20.0])
    X = np.diag(1.0 / sds)
    yv = np.zeros(3)
    res = [orc.nuts(X, None, step_size=0.01, max_tree_depth=10, num_warmup=600, num_samples=800,
                    seed=21, chain=c, prior_scale=1e6, target=orc.TARGET_LINGAUSS, yv=yv,
                    noise_scale=1.0, adapt_diag_mass=True, adapt_step_size=True)
           for c in range(3)]
    for r in res:
        np.testing.assert_allclose(r["inv_mass"], sds**2, rtol=0.35)
    S = np.stack([r["samples"] for r in res])
    flat = S.reshape(-1, 3)
    ess_m = ess_columns(S)
    mcse = flat.std(axis=0, ddof=1) / np.sqrt(ess_m)
    assert (np.abs(flat.mean(0)) < 4 * mcse).all()
    sq = S**2
    ess_v = ess_columns(sq)
    mcse_v = sq.reshape(-1, 3).std(axis=0, ddof=1) / np.sqrt(ess_v)
    assert (np.abs(sq.reshape(-1, 3).mean(0) - sds**2) < 4 * mcse_v).all()
    # with the metric adapted the trees stay shallow despite the 400:1 scales
    depth = np.concatenate([r["stats"]["tree_depth"] for r in res])
    assert depth.mean() < 4.0


def test_fixed_step_unchanged_by_adaptation_code(orc):
    # without the adaptation flag the step size is the given one
    X, y, _ = workloads.make_logistic(30, 3, w_scale=1.0, key=5)
    r = orc.nuts(X, y, step_size=0.123, max_tree_depth=5, num_warmup=20, num_samples=5, seed=1)
    assert r["step_size"] == 0.123
