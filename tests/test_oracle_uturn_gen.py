"""Pins for the oracle's generalised U-turn criterion (reading R20): the
recursive builder, where the momentum sum of a subtree is literally the sum
of its two halves' sums at every merge, and the iterative builder, where it
is a difference of running sums kept in the checkpoint slots, make the same
trees and proposals under the same draws; the criterion changes decisions
relative to the endpoint one; and sampling with it stays exact (conjugate
Gaussian within 4 Monte Carlo standard errors)."""
import numpy as np
import pytest

import workloads
from oracle.ess import ess_columns

CASES = [(0.3, 6), (0.8, 8), (6.0, 6), (1e-3, 5)]


def _tiny(seed, N, D):
    X, y, _ = workloads.make_logistic(N, D, w_scale=1.5, key=[100, seed])
    return X, y


def test_generalised_definition(orc):
    # Betancourt (2017), App. A.4.2: a trajectory turns when the momentum at
    # either end, pushed through the inverse metric, no longer has a positive
    # projection onto the trajectory's momentum sum
    r = np.array([1.0, 0.0])
    assert orc.is_uturn_generalized(r, [1.0, 0.2], [-1.0, 0.0])      # one end turned
    assert orc.is_uturn_generalized(r, [-1.0, 0.0], [1.0, 0.2])
    assert not orc.is_uturn_generalized(r, [1.0, 5.0], [0.5, -3.0])  # both still forward
    assert orc.is_uturn_generalized(r, [0.0, 1.0], [2.0, 0.0])       # a zero projection turns
    # the inverse metric weights the projection: rho . M^-1 p
    rho, pa, pb = np.array([1.0, 1.0]), np.array([1.0, -0.5]), np.array([1.0, 1.0])
    assert not orc.is_uturn_generalized(rho, pa, pb, inv_mass=[1.0, 1.0])
    assert orc.is_uturn_generalized(rho, pa, pb, inv_mass=[1.0, 4.0])


@pytest.mark.parametrize("eps,maxd", CASES)
def test_recursive_equals_iterative_generalised(orc, eps, maxd):
    turned = 0
    for seed in range(30):
        N, D = 5 + seed % 16, 1 + seed % 3
        X, y = _tiny(seed, N, D)
        kw = dict(step_size=eps, max_tree_depth=maxd, num_warmup=5, num_samples=15, seed=seed,
                  chain=seed % 3, trace_cap=1 << 14, inv_mass=np.linspace(0.5, 1.5, D),
                  uturn_generalized=True)
        a = orc.nuts(X, y, builder=orc.BUILDER_ITERATIVE, **kw)
        b = orc.nuts(X, y, builder=orc.BUILDER_RECURSIVE, **kw)
        assert np.array_equal(a["samples"], b["samples"])
        assert a["stats"].tobytes() == b["stats"].tobytes()
        assert np.array_equal(a["trace"], b["trace"])
        turned += int(a["stats"]["turning"].sum())
    if 1e-3 < eps < 6.0:
        assert turned > 0


def test_criterion_changes_decisions(orc):
    diff = 0
    for seed in range(20):
        X, y = _tiny(seed, 30, 2)
        kw = dict(step_size=0.3, max_tree_depth=8, num_warmup=0, num_samples=40, seed=seed)
        a = orc.nuts(X, y, **kw)
        b = orc.nuts(X, y, uturn_generalized=True, **kw)
        diff += int((a["stats"]["num_steps"] != b["stats"]["num_steps"]).sum())
    assert diff > 0


@pytest.mark.slow
def test_generalised_conjugate_gaussian(orc):
    X, yv = workloads.make_lingauss(30, 3, key=21, noise_scale=0.5)
    s, sn = 2.0, 0.5
    P = X.T @ X / sn**2 + np.eye(3) / s**2
    Sigma = np.linalg.inv(P)
    mu = Sigma @ X.T @ yv / sn**2
    runs = [orc.nuts(X, None, step_size=0.05, max_tree_depth=8, num_warmup=200, num_samples=2000,
                     seed=1, chain=c, prior_scale=s, target=orc.TARGET_LINGAUSS, yv=yv,
                     noise_scale=sn, uturn_generalized=True) for c in range(4)]
    S = np.stack([r["samples"] for r in runs])
    flat = S.reshape(-1, 3)
    mcse = flat.std(axis=0, ddof=1) / np.sqrt(ess_columns(S))
    assert (np.abs(flat.mean(0) - mu) < 4 * mcse).all()
    sq = (S - mu) ** 2
    mcse_v = sq.reshape(-1, 3).std(axis=0, ddof=1) / np.sqrt(ess_columns(sq))
    assert (np.abs(sq.reshape(-1, 3).mean(0) - np.diag(Sigma)) < 4 * mcse_v).all()
    # the criterion still stops trajectories well short of the depth limit
    depth = np.concatenate([r["stats"]["tree_depth"] for r in runs])
    assert depth.mean() < 7.0
