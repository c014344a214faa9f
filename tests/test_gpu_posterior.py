"""Statistical acceptance of long GPU runs: posterior moments against the
oracle's normal approximation of the same posterior (Appendix B model).

Decision-by-decision parity covers tens of iterations; in fp32 a decision
can flip once a uniform falls within the fp32 energy error of its threshold,
after which two correct chains part ways.  These tests check what must still
hold: the draws of the full protocol (warmup then samples, Section 4's
covtype runs) have posterior means within 4 Monte Carlo standard errors of
the oracle's skewness-corrected Laplace mean (error of order 1/N^2, far
below the MCSE at these N), and variances within 4 MCSE of the Laplace
covariance's diagonal (error of order 1/N).  MCSE = sd / sqrt(ESS), ESS by
Geyer's initial monotone sequence (pooled over chains that share a target).
The oracle runs on the fp32-rounded X promoted to fp64 (reading R11).

For the 4,096 independent small models every chain is its own posterior:
the z-scores of all 4,096 x 9 means against each chain's own corrected
Laplace mean must look standard normal (Kolmogorov-Smirnov).
"""
import numpy as np
import pytest
from scipy import stats

import workloads
from oracle.ess import ess_columns
from tests.gpu_common import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sampler():
    import paper_1912_11554_amd as nuts
    return nuts.Sampler(0)


def _z_scores(samples, lap):
    """z of the pooled mean against the corrected Laplace mean and of the
    pooled variance against the Laplace variances, per coordinate."""
    S = np.asarray(samples)
    if S.ndim == 2:
        S = S[None]
    flat = S.reshape(-1, S.shape[-1])
    m = flat.mean(axis=0)
    mcse = flat.std(axis=0, ddof=1) / np.sqrt(ess_columns(S))
    sq = (S - m) ** 2
    sqf = sq.reshape(-1, S.shape[-1])
    mcse_v = sqf.std(axis=0, ddof=1) / np.sqrt(ess_columns(sq))
    z_m = (m - lap["mean"]) / mcse
    z_v = (sqf.mean(axis=0) - np.diag(lap["cov"])) / mcse_v
    return z_m, z_v


def test_covtype_f32_full_protocol_within_4_mcse(sampler, orc):
    # the metric's workload as the paper runs it: 1000 warmup + 1000 draws,
    # fp32 X on the grid path
    wl = workloads.WORKLOADS["covtype_n581012_d55_f32"]
    X, y = workloads.make_workload(wl)
    say("posterior covtype f32", wl.num_warmup, "+", wl.num_samples)
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=wl.num_warmup, num_samples=wl.num_samples, seed=wl.seed, path=2)
    assert int(r["stats"]["diverging"].sum()) == 0
    lap = orc.logistic_laplace(X, y, wl.prior_scale)
    z_m, z_v = _z_scores(r["samples"], lap)
    say("covtype f32 max |z| mean", np.abs(z_m).max(), "variance", np.abs(z_v).max())
    assert np.all(np.abs(z_m) < 4.0), np.argmax(np.abs(z_m))
    assert np.all(np.abs(z_v) < 4.0), np.argmax(np.abs(z_v))


def test_shared256_f32_pooled_chains_within_4_mcse(sampler, orc):
    # 256 chains on one 200,000 x 129 fp32 data set, the matrix-core batch
    # path, 500 warmup + 500 draws each, pooled
    wl = workloads.WORKLOADS["shared256_n200000_d129_f32"]
    X, y = workloads.make_workload(wl)
    say("posterior shared256 f32", wl.num_chains, "chains")
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=wl.num_warmup, num_samples=wl.num_samples,
                       num_chains=wl.num_chains, seed=wl.seed, path=3)
    assert int(r["stats"]["diverging"].sum()) == 0
    lap = orc.logistic_laplace(X, y, wl.prior_scale)
    z_m, z_v = _z_scores(r["samples"], lap)
    say("shared256 max |z| mean", np.abs(z_m).max(), "variance", np.abs(z_v).max())
    assert np.all(np.abs(z_m) < 4.0), np.argmax(np.abs(z_m))
    assert np.all(np.abs(z_v) < 4.0), np.argmax(np.abs(z_v))


def test_chains4096_z_scores_standard_normal(sampler, orc):
    # 4,096 chains, each with its own 500 x 9 data set, one wavefront per
    # chain, 500 warmup + 500 draws; every chain against its own posterior
    wl = workloads.WORKLOADS["chains4096_n500_d9_f64"]
    C = wl.num_chains
    X, y = workloads.make_workload(wl)
    say("posterior chains4096", C, "chains")
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=wl.num_warmup, num_samples=wl.num_samples, num_chains=C,
                       seed=wl.seed, per_chain=True)
    z = np.empty((C, wl.D))
    for c in range(C):
        lap = orc.logistic_laplace(X[c], y[c], wl.prior_scale)
        z[c] = _z_scores(r["samples"][c], lap)[0]
    z = z.ravel()
    ks = stats.kstest(z, "norm")
    say("chains4096 z mean", z.mean(), "sd", z.std(), "KS", ks.statistic, ks.pvalue)
    assert ks.pvalue > 1e-3, ks
    assert abs(z.mean()) < 0.05
    assert 0.95 < z.std() < 1.05
