"""GPU parity of the fused potential + gradient kernel against the oracle.

Bar: fp64 X -- relative error <= 1e-10 for U, and for the gradient both
normwise, max_j |g_j - g_ref_j| <= 1e-10 max_j |g_ref_j|, and per component
relative to the magnitude of the summed terms; fp32 X -- the same
comparisons against the oracle run on the fp32-rounded X promoted to fp64,
bar 1e-4 (the kernel accumulates in fp64, so it lands far inside it).
"""
import numpy as np
import pytest

import workloads
from tests.gpu_common import grad_tol, say

pytestmark = pytest.mark.gpu

RTOL = {"f64": 1e-10, "f32": 1e-4}


@pytest.fixture(scope="module")
def sampler():
    import paper_1912_11554_amd as nuts
    return nuts.Sampler(0)


def _check(sampler, orc, X, y, w, s, dt):
    say("potential_grad", X.shape, dt, "s", s)
    U, g = sampler.potential_grad(X, y, w, prior_scale=s)
    U_ref, g_ref = orc.logistic_potential_grad(X.astype(np.float64), y, w, prior_scale=s)
    assert abs(U - U_ref) <= RTOL[dt] * abs(U_ref), (U, U_ref)
    tol = grad_tol(X, w, g_ref, s, RTOL[dt])
    assert (np.abs(g - g_ref) <= tol).all(), np.max(np.abs(g - g_ref) / tol)
    assert np.abs(g - g_ref).max() <= RTOL[dt] * np.abs(g_ref).max(), (
        np.abs(g - g_ref).max() / np.abs(g_ref).max())
    return abs(U - U_ref) / abs(U_ref)


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("N,D", [(1, 1), (63, 2), (64, 5), (65, 11), (1000, 11), (4097, 9),
                                 (777, 33), (3000, 55), (130, 63), (500, 64), (301, 65),
                                 (1000, 129), (777, 200), (513, 257), (200, 320),
                                 (301, 288), (299, 289), (203, 319)])
def test_random_positions(sampler, orc, dt, N, D):
    X, y, w_true = workloads.make_logistic(N, D, w_scale=0.7, key=[50, N * 1000 + D],
                                           dtype=dt)
    rng = np.random.default_rng(N * 100 + D)
    for w in (np.zeros(D), w_true, w_true + rng.normal(size=D)):
        _check(sampler, orc, X, y, w, 1.0, dt)
    _check(sampler, orc, X, y, w_true, 2.5, dt)


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_saturating_logits(sampler, orc, dt):
    # |eta| > 40 on most rows: exp(-|t|) underflows towards 0 without loss
    X, y, w_true = workloads.make_logistic(500, 7, w_scale=1.0, key=51, dtype=dt)
    w = 40.0 * np.sign(w_true) + w_true
    _check(sampler, orc, X, y, w, 1.0, dt)
    _check(sampler, orc, X, y, -w, 1.0, dt)


def test_prior_only(sampler, orc):
    w = np.array([0.3, -1.2, 2.0])
    X = np.zeros((0, 3))
    y = np.zeros(0, dtype=np.uint8)
    say("potential_grad N=0")
    U, g = sampler.potential_grad(X, y, w, prior_scale=1.5)
    U_ref, g_ref = orc.logistic_potential_grad(X, y, w, prior_scale=1.5)
    assert abs(U - U_ref) <= 1e-14 * abs(U_ref)
    np.testing.assert_allclose(g, g_ref, rtol=1e-15)


def test_batched_shared_and_per_chain(sampler, orc):
    # K positions on one data set, and K data sets with one position each
    X, y, w_true = workloads.make_logistic(2000, 10, w_scale=1.0, key=52)
    rng = np.random.default_rng(5)
    W = w_true + 0.3 * rng.normal(size=(17, 10))
    say("potential_grad batched shared K=17")
    d = sampler.data(X, y)
    U, G = d.potential_grad(W)
    d.free()
    for k in range(17):
        U_ref, g_ref = orc.logistic_potential_grad(X, y, W[k])
        assert abs(U[k] - U_ref) <= 1e-10 * abs(U_ref)
        assert (np.abs(G[k] - g_ref) <= grad_tol(X, W[k], g_ref, 1.0, 1e-10)).all()
        assert np.abs(G[k] - g_ref).max() <= 1e-10 * np.abs(g_ref).max()
    wl = workloads.WORKLOADS["chains4096_n500_d9_f64"]
    Xc, yc = workloads.make_workload(wl, chains=range(40))
    Wc = rng.normal(size=(40, 9))
    say("potential_grad per-chain K=40")
    d = sampler.data(Xc, yc, per_chain=True)
    U, G = d.potential_grad(Wc)
    d.free()
    for k in range(40):
        U_ref, g_ref = orc.logistic_potential_grad(Xc[k], yc[k], Wc[k])
        assert abs(U[k] - U_ref) <= 1e-10 * abs(U_ref)
        assert (np.abs(G[k] - g_ref) <= grad_tol(Xc[k], Wc[k], g_ref, 1.0, 1e-10)).all()
        assert np.abs(G[k] - g_ref).max() <= 1e-10 * np.abs(g_ref).max()


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("N,D,K,per_chain", [(1, 1, 64, True), (77, 8, 100, True), (130, 9, 4096, True),
                                             (500, 16, 300, False), (1000, 17, 64, True),
                                             (257, 32, 70, False), (511, 33, 129, True),
                                             (500, 64, 65, True), (4000, 55, 64, False)])
def test_many_small_items(sampler, orc, dt, N, D, K, per_chain):
    # many positions on data sets of at most 32 row blocks (D <= 64): one
    # wavefront an item; per-chain data sets or one shared set, ragged row
    # counts, every item compared with the oracle
    rng = np.random.default_rng(N * 7 + D + K)
    if per_chain:
        nsets = K if K <= 130 else 130
        sets = [workloads.make_logistic(N, D, w_scale=0.7, key=[76, (N * 1000 + D) * 1000 + c], dtype=dt)[:2]
                for c in range(nsets)]
        idx = np.arange(K) % nsets
        X = np.stack([sets[i][0] for i in idx])
        y = np.stack([sets[i][1] for i in idx])
    else:
        X, y, _ = workloads.make_logistic(N, D, w_scale=0.7, key=[77, N * 1000 + D], dtype=dt)
    W = 0.5 * rng.normal(size=(K, D))
    say("potential_grad many items", N, D, K, per_chain, dt)
    d = sampler.data(X, y, per_chain=per_chain)
    U, G = d.potential_grad(W)
    d.free()
    for k in range(K):
        Xk, yk = (X[k], y[k]) if per_chain else (X, y)
        U_ref, g_ref = orc.logistic_potential_grad(Xk.astype(np.float64), yk, W[k])
        assert abs(U[k] - U_ref) <= RTOL[dt] * abs(U_ref), (k, U[k], U_ref)
        assert (np.abs(G[k] - g_ref) <= grad_tol(Xk, W[k], g_ref, 1.0, RTOL[dt])).all(), k
        assert np.abs(G[k] - g_ref).max() <= RTOL[dt] * np.abs(g_ref).max(), k


@pytest.mark.parametrize("name", ["covtype_n581012_d55_f64", "covtype_n581012_d55_f32"])
def test_full_size_covtype(sampler, orc, name):
    wl = workloads.WORKLOADS[name]
    X, y = workloads.make_workload(wl)
    rng = np.random.default_rng(7)
    _, _, w_true = workloads.make_logistic(1, wl.D, w_scale=wl.w_scale, key=wl.data_seed)
    for w in (np.zeros(wl.D), w_true + 0.01 * rng.normal(size=wl.D)):
        _check(sampler, orc, X, y, w, 1.0, wl.dtype)


def test_full_size_streaming(sampler, orc):
    # the 4,000,000 x 257 fp32 set (4.1 GB, 10 % of the features zero) of
    # the streaming workload, at zero and near its generating weights; the
    # oracle promotes the fp32 rows to fp64 one at a time
    wl = workloads.WORKLOADS["stream_n4m_d257_f32"]
    X, y = workloads.make_workload(wl)
    _, _, w_true = workloads.make_logistic(1, wl.D, w_scale=wl.w_scale, key=wl.data_seed)
    colsum = np.abs(X).sum(axis=0, dtype=np.float64)
    d = sampler.data(X, y)
    rng = np.random.default_rng(8)
    for w in (np.zeros(wl.D), w_true + 0.01 * rng.normal(size=wl.D)):
        say("potential_grad full-size streaming", X.shape)
        U, G = d.potential_grad(w[None, :])
        U_ref, g_ref = orc.logistic_potential_grad_f32(X, y, w)
        assert abs(U[0] - U_ref) <= RTOL["f32"] * abs(U_ref), (U[0], U_ref)
        tol = RTOL["f32"] * (np.abs(g_ref) + colsum + np.abs(w) + 1.0)
        assert (np.abs(G[0] - g_ref) <= tol).all(), np.max(np.abs(G[0] - g_ref) / tol)
        assert np.abs(G[0] - g_ref).max() <= RTOL["f32"] * np.abs(g_ref).max()
    d.free()


def test_errors_are_reported(sampler):
    import paper_1912_11554_amd as nuts
    X = np.zeros((10, 3))
    y = np.zeros(10, dtype=np.uint8)
    y[3] = 2
    say("error paths")
    with pytest.raises(nuts.NutsError) as e:
        sampler.potential_grad(X, y, np.zeros(3))
    assert e.value.code == nuts.NUTS_EINVAL
    with pytest.raises(nuts.NutsError) as e:
        sampler.potential_grad(np.zeros((10, 3)), np.zeros(10, np.uint8), np.zeros(3),
                               prior_scale=-1.0)
    assert e.value.code == nuts.NUTS_EINVAL
    with pytest.raises(nuts.NutsError) as e:
        sampler.potential_grad(np.zeros((10, 400)), np.zeros(10, np.uint8), np.zeros(400))
    assert e.value.code == nuts.NUTS_EUNSUPPORTED
