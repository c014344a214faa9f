"""Pins for the oracle's semi-supervised HMM potential (reading R21): the
forward algorithm against brute-force enumeration of the hidden paths, the
additive-log-ratio Jacobian against a numerical log-determinant, the
hand-derived adjoint against central differences, and the sampler's two
tree builders agreeing on this target."""
import itertools

import numpy as np
import pytest

import workloads


def _rows(q, K, V):
    nt = K * (K - 1)
    sm = lambda a: np.exp(np.append(a, 0.0) - np.logaddexp.reduce(np.append(a, 0.0)))
    th = np.array([sm(q[j * (K - 1):(j + 1) * (K - 1)]) for j in range(K)])
    ph = np.array([sm(q[nt + k * (V - 1):nt + (k + 1) * (V - 1)]) for k in range(K)])
    return th, ph


def _log_jac(a):
    """log |det d x[:-1] / d a| of x = softmax(a, 0), by central differences."""
    n = a.size
    J = np.zeros((n, n))
    for i in range(n):
        e = np.zeros(n)
        e[i] = 1e-6
        xp = np.exp(np.append(a + e, 0) - np.logaddexp.reduce(np.append(a + e, 0)))[:-1]
        xm = np.exp(np.append(a - e, 0) - np.logaddexp.reduce(np.append(a - e, 0)))[:-1]
        J[:, i] = (xp - xm) / 2e-6
    return np.linalg.slogdet(J)[1]


@pytest.mark.parametrize("Tsup", [0, 1, 3])
def test_forward_equals_enumeration(orc, Tsup):
    K, V, Tu = 3, 4, 6
    rng = np.random.default_rng(Tsup)
    w = rng.integers(0, V, size=Tsup + Tu).astype(np.uint8)
    z = rng.integers(0, K, size=Tsup).astype(np.uint8)
    q = rng.normal(0, 0.8, size=orc.hmm_dim(K, V))
    U, _ = orc.hmm_potential_grad(w, z, K, V, q)
    th, ph = _rows(q, K, V)
    f = np.log(th).sum() + np.log(ph).sum()
    f += sum(np.log(ph[z[t], w[t]]) for t in range(Tsup))
    f += sum(np.log(th[z[t - 1], z[t]]) for t in range(1, Tsup))
    tot = 0.0
    for path in itertools.product(range(K), repeat=Tu):
        p = 1.0
        for s, k in enumerate(path):
            if s == 0:
                p *= th[z[-1], k] if Tsup > 0 else 1.0 / K
            else:
                p *= th[path[s - 1], k]
            p *= ph[k, w[Tsup + s]]
        tot += p
    f += np.log(tot)
    np.testing.assert_allclose(U, -f, rtol=1e-12)


def test_jacobian_is_log_determinant(orc):
    # no data: U = -(sum of the rows' log |Jacobian|)
    K, V = 3, 5
    q = np.random.default_rng(7).normal(0, 1.0, size=orc.hmm_dim(K, V))
    U, _ = orc.hmm_potential_grad(np.zeros(0, np.uint8), np.zeros(0, np.uint8), K, V, q)
    nt = K * (K - 1)
    want = sum(_log_jac(q[j * (K - 1):(j + 1) * (K - 1)]) for j in range(K))
    want += sum(_log_jac(q[nt + k * (V - 1):nt + (k + 1) * (V - 1)]) for k in range(K))
    np.testing.assert_allclose(U, -want, rtol=1e-7)


@pytest.mark.parametrize("Tsup", [0, 100])
def test_gradient_central_differences(orc, Tsup):
    w, z, _, _ = workloads.make_hmm(T=600, Tsup=Tsup, key=8)
    K, V = 3, 10
    q = np.random.default_rng(9).normal(0, 0.5, size=orc.hmm_dim(K, V))
    _, g = orc.hmm_potential_grad(w, z, K, V, q)
    h = 1e-5
    fd = np.zeros_like(q)
    for i in range(q.size):
        e = np.zeros_like(q)
        e[i] = h
        fd[i] = (orc.hmm_potential_grad(w, z, K, V, q + e)[0]
                 - orc.hmm_potential_grad(w, z, K, V, q - e)[0]) / (2 * h)
    np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-6)


def test_builders_agree_on_hmm(orc):
    w, z, _, _ = workloads.make_hmm(T=120, Tsup=20, key=10)
    hmm = dict(w=w, z=z, K=3, V=10)
    kw = dict(step_size=0.1, max_tree_depth=6, num_warmup=3, num_samples=10, seed=2, hmm=hmm,
              trace_cap=1 << 14)
    a = orc.nuts(None, None, builder=orc.BUILDER_ITERATIVE, **kw)
    b = orc.nuts(None, None, builder=orc.BUILDER_RECURSIVE, **kw)
    assert np.array_equal(a["samples"], b["samples"])
    assert a["stats"].tobytes() == b["stats"].tobytes()
    assert a["stats"]["num_steps"].sum() > 10
