"""Pins for the oracle's leapfrog integrator (kick-drift-kick, one gradient
per step): time reversibility, volume preservation, O(eps^2) energy error,
and the exact linear propagator on a quadratic potential."""
import numpy as np
import pytest

import workloads


def _logistic(N=200, D=4, seed=9):
    X, y, w = workloads.make_logistic(N, D, w_scale=1.0, key=seed)
    return X, y, w


def test_reversibility(orc):
    X, y, w = _logistic()
    rng = np.random.default_rng(0)
    im = rng.uniform(0.5, 2.0, size=4)
    q0 = w + 0.2 * rng.normal(size=4)
    p0 = rng.normal(size=4)
    for h, L in ((0.01, 200), (0.05, 50)):
        q1, p1, _ = orc.leapfrog(X, y, q0, p0, h, L, inv_mass=im)
        q2, p2, _ = orc.leapfrog(X, y, q1, -p1, h, L, inv_mass=im)
        np.testing.assert_allclose(q2, q0, rtol=1e-12, atol=1e-12 * np.abs(q0).max())
        np.testing.assert_allclose(-p2, p0, rtol=1e-12, atol=1e-12 * np.abs(p0).max())


def test_volume_preservation(orc):
    # the leapfrog map is symplectic: its Jacobian has determinant 1
    X, y, w = _logistic(N=150, D=3, seed=10)
    rng = np.random.default_rng(1)
    q0, p0 = w + 0.3 * rng.normal(size=3), rng.normal(size=3)
    h, L, d = 0.05, 10, 1e-6
    x0 = np.concatenate([q0, p0])

    def flow(x):
        q, p, _ = orc.leapfrog(X, y, x[:3], x[3:], h, L)
        return np.concatenate([q, p])

    J = np.zeros((6, 6))
    for k in range(6):
        e = np.zeros(6)
        e[k] = d
        J[:, k] = (flow(x0 + e) - flow(x0 - e)) / (2 * d)
    assert np.linalg.det(J) == pytest.approx(1.0, abs=1e-6)


def _energy(orc, X, y, q, p, im):
    U, _ = orc.logistic_potential_grad(X, y, q)
    return U + 0.5 * np.sum(im * p * p)


def test_energy_error_second_order(orc):
    X, y, w = _logistic(N=300, D=5, seed=11)
    rng = np.random.default_rng(2)
    im = np.ones(5)
    q0, p0 = w + 0.1 * rng.normal(size=5), rng.normal(size=5)
    H0 = _energy(orc, X, y, q0, p0, im)
    T = 0.8
    hs, errs = [], []
    for k in range(5):
        h = 0.04 / 2**k
        L = int(round(T / h))
        q1, p1, _ = orc.leapfrog(X, y, q0, p0, h, L)
        hs.append(h)
        errs.append(abs(_energy(orc, X, y, q1, p1, im) - H0))
    slope = np.polyfit(np.log(hs), np.log(errs), 1)[0]
    assert slope == pytest.approx(2.0, abs=0.15)


def test_quadratic_exact_propagator(orc):
    # U = omega^2 q^2 / 2 via the linear-Gaussian target with one row x = a,
    # response 0, noise sn, prior s: omega^2 = a^2 / sn^2 + 1 / s^2.  The
    # leapfrog step is then the linear map
    #   [[1 - x/2, h mu], [-h omega^2 (1 - x/4), 1 - x/2]],  x = h^2 mu omega^2.
    a, sn, s, mu, h, L = 3.0, 0.5, 2.0, 0.7, 0.1, 37
    om2 = a * a / (sn * sn) + 1.0 / (s * s)
    x = h * h * mu * om2
    M = np.array([[1 - x / 2, h * mu], [-h * om2 * (1 - x / 4), 1 - x / 2]])
    assert np.linalg.det(M) == pytest.approx(1.0, abs=1e-14)
    want = np.linalg.matrix_power(M, L) @ np.array([0.8, -0.3])
    q, p, _ = orc.leapfrog(np.array([[a]]), None, np.array([0.8]), np.array([-0.3]), h, L,
                           inv_mass=np.array([mu]), prior_scale=s,
                           target=orc.TARGET_LINGAUSS, yv=np.array([0.0]), noise_scale=sn)
    np.testing.assert_allclose([q[0], p[0]], want, rtol=1e-12)
