"""Pins for the oracle's merge-structured subtree proposals (reading R22):
the recursive builder, which merges the two halves of every subtree
literally, and the iterative builder, which keeps one completed block per
level and merges like a binary counter, make the same trees and proposals
under the same draws; the variant draws differently from the streaming
choice; and it selects each trajectory point with the exact multinomial /
biased-progressive probability (chi-square over re-drawn selections on a
fixed trajectory), so sampling stays exact (conjugate Gaussian)."""
import numpy as np
import pytest

import workloads
from oracle.ess import ess_columns
from tests.test_oracle_nuts import _GAUSS, _SDS, _exact_selection

CASES = [(0.3, 6), (0.8, 8), (6.0, 6), (1e-3, 5)]


def _tiny(seed, N, D):
    X, y, _ = workloads.make_logistic(N, D, w_scale=1.5, key=[101, seed])
    return X, y


@pytest.mark.parametrize("eps,maxd", CASES)
@pytest.mark.parametrize("gen", [False, True])
def test_recursive_equals_iterative_submerge(orc, eps, maxd, gen):
    stopped = 0
    for seed in range(25):
        N, D = 5 + seed % 16, 1 + seed % 3
        X, y = _tiny(seed, N, D)
        kw = dict(step_size=eps, max_tree_depth=maxd, num_warmup=5, num_samples=15, seed=seed,
                  chain=seed % 3, trace_cap=1 << 14, inv_mass=np.linspace(0.5, 1.5, D),
                  uturn_generalized=gen, subtree_merge=True)
        a = orc.nuts(X, y, builder=orc.BUILDER_ITERATIVE, **kw)
        b = orc.nuts(X, y, builder=orc.BUILDER_RECURSIVE, **kw)
        assert np.array_equal(a["samples"], b["samples"])
        assert a["stats"].tobytes() == b["stats"].tobytes()
        assert np.array_equal(a["trace"], b["trace"])
        stopped += int((a["stats"]["turning"] | a["stats"]["diverging"]).sum())
    assert stopped > 0


def test_variant_draws_differently(orc):
    # same trajectories (the tree decisions do not depend on the selection
    # draws within an iteration), different proposals
    diff = 0
    for seed in range(10):
        X, y = _tiny(seed, 30, 2)
        kw = dict(step_size=0.3, max_tree_depth=8, num_warmup=0, num_samples=1, seed=seed,
                  init_q=np.array([0.2, -0.1]))
        a = orc.nuts(X, y, **kw)
        b = orc.nuts(X, y, subtree_merge=True, **kw)
        assert a["stats"]["num_steps"][0] == b["stats"]["num_steps"][0]
        diff += int(a["stats"]["proposal_index"][0] != b["stats"]["proposal_index"][0])
    assert diff > 0


@pytest.mark.slow
@pytest.mark.parametrize("eps,seed", [(0.3, 2), (0.35, 0)])
def test_selection_distribution_submerge(orc, eps, seed):
    # over a fixed trajectory, re-drawing only the selection uniforms must
    # reproduce the exact selection probabilities (chi-square test)
    from scipy import stats as sst
    X, y = np.diag(1.0 / _SDS), None
    q0 = np.array([0.1, 2.0])
    kw = dict(step_size=eps, max_tree_depth=6, seed=seed, subtree_merge=True, **_GAUSS)

    def one(salt):
        return orc.nuts(X, y, num_warmup=0, num_samples=1, init_q=q0, first_iter=7,
                        leaves_cap=4096, sel_salt=salt, **kw)

    ref = one(0)
    prob = _exact_selection(ref["leaves"], ref["stats"][0])
    counts = {}
    R = 12000
    for salt in range(1, R + 1):
        r = one(salt)
        k = int(r["stats"]["proposal_index"][0])
        counts[k] = counts.get(k, 0) + 1
    assert set(counts) <= set(prob)
    keys = sorted(prob)
    obs = np.array([counts.get(k, 0) for k in keys], dtype=float)
    exp = np.array([prob[k] for k in keys]) * R
    assert len(keys) >= 4
    order = np.argsort(exp)
    o2, e2, acc_o, acc_e = [], [], 0.0, 0.0
    for i in order:
        acc_o += obs[i]
        acc_e += exp[i]
        if acc_e >= 5:
            o2.append(acc_o)
            e2.append(acc_e)
            acc_o = acc_e = 0.0
    if acc_e > 0:
        o2[-1] += acc_o
        e2[-1] += acc_e
    assert sst.chisquare(o2, e2).pvalue > 1e-4


@pytest.mark.slow
def test_submerge_conjugate_gaussian(orc):
    X, yv = workloads.make_lingauss(30, 3, key=21, noise_scale=0.5)
    s, sn = 2.0, 0.5
    P = X.T @ X / sn**2 + np.eye(3) / s**2
    Sigma = np.linalg.inv(P)
    mu = Sigma @ X.T @ yv / sn**2
    runs = [orc.nuts(X, None, step_size=0.05, max_tree_depth=8, num_warmup=200, num_samples=2000,
                     seed=3, chain=c, prior_scale=s, target=orc.TARGET_LINGAUSS, yv=yv,
                     noise_scale=sn, subtree_merge=True) for c in range(4)]
    S = np.stack([r["samples"] for r in runs])
    flat = S.reshape(-1, 3)
    mcse = flat.std(axis=0, ddof=1) / np.sqrt(ess_columns(S))
    assert (np.abs(flat.mean(0) - mu) < 4 * mcse).all()
    sq = (S - mu) ** 2
    mcse_v = sq.reshape(-1, 3).std(axis=0, ddof=1) / np.sqrt(ess_columns(sq))
    assert (np.abs(sq.reshape(-1, 3).mean(0) - np.diag(Sigma)) < 4 * mcse_v).all()
