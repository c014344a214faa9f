"""GPU parity of the warmup adaptation (NUTS_ADAPT_STEP_SIZE, with and
without the windowed diagonal mass) against the oracle.

Bar (fp64): the step-size heuristic, every dual-averaging update and the
window ends run the same arithmetic on both sides, but the device's exp,
log and pow, its fused multiply-adds and its wave-order sums may differ from
the host's in the last bit.  Tree decisions are bit-exact.  The continuous
results are compared within a bar set by the oracle itself: the same run
with every element of X moved by one ulp changes the adapted step size and
the samples by some amount s (about 1e-12 with the step size alone; 1e-10
to 1e-5 once the windowed mass feeds sample variances from a few dozen
draws back into the metric), and the GPU must agree to max(1e-9, 100 s).  fp32 data on the matrix-core
path: decisions bit-exact over a short warmup; there the row terms run in
fp32, so each energy carries an error of about 1e-7 of the summed row losses
(~3e-6 absolute here), the accept statistics move by as much, and the dual
averaging multiplies their differences by up to sqrt(m)/gamma ~ 60: the
step size and the samples are held to 2e-4.
"""
import numpy as np
import pytest

import workloads
from tests.gpu_common import DECISION_FIELDS, compare_chain, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sampler():
    import paper_1912_11554_amd as nuts
    return nuts.Sampler(0)


def _bar(orc, X, y, ref, **kw):
    """max(1e-9, 100 s), s the oracle's own largest relative change (step
    size, inverse mass, samples) when every element of X moves by one ulp in
    a random direction, over two such draws: the GPU's last-bit differences
    are spread over all of its arithmetic in the same way."""
    rng = np.random.default_rng(1234)
    s = 0.0
    for _ in range(2):
        X64 = np.asarray(X, dtype=np.float64)
        Xp = np.nextafter(X64, rng.choice([-np.inf, np.inf], size=X64.shape))
        b = orc.nuts(Xp, y, **kw)
        s = max(s, abs(b["step_size"] / ref["step_size"] - 1.0),
                np.max(np.abs(b["inv_mass"] / ref["inv_mass"] - 1.0)),
                np.max(np.abs(b["samples"] - ref["samples"]) / (1.0 + np.abs(ref["samples"]))))
    return max(1e-9, 100.0 * s)


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("mass", [False, True])
def test_adaptation_matches_oracle(sampler, orc, path, mass):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    W, S = 200, 40
    say("adapt logreg_n1000_d11 path", path, "mass", mass)
    kw = dict(step_size=0.3, max_tree_depth=wl.max_tree_depth, num_warmup=W, num_samples=S,
              seed=wl.seed, adapt_diag_mass=mass)
    r = sampler.sample(X, y, path=path, adapt_step_size=True, target_accept=0.8, **kw)
    ref = orc.nuts(X, y, adapt_step_size=True, target_accept=0.8, **kw)
    tol = _bar(orc, X, y, ref, adapt_step_size=True, target_accept=0.8, **kw)
    np.testing.assert_allclose(r["step_size"][0], ref["step_size"], rtol=tol)
    assert ref["step_size"] != 0.3
    np.testing.assert_allclose(r["inv_mass"][0], ref["inv_mass"], rtol=tol)
    if mass:
        assert not np.allclose(ref["inv_mass"], 1.0)
    compare_chain(r["samples"][0], r["stats"][0], ref, atol=tol)
    assert r["grad_evals"] == ref["grad_evals"]


def test_adaptation_edge_cases(sampler, orc):
    # warmup of one iteration (heuristic, one update, then the average);
    # warmup too short for mass windows; a start step far too large
    X, y, _ = workloads.make_logistic(300, 5, w_scale=1.0, key=[62, 1])
    for W, eps0, mass in [(1, 0.01, False), (15, 0.01, True), (30, 25.0, True)]:
        say("adapt edge", W, eps0, mass)
        kw = dict(step_size=eps0, max_tree_depth=8, num_warmup=W, num_samples=10, seed=3,
                  adapt_diag_mass=mass)
        r = sampler.sample(X, y, path=1, adapt_step_size=True, **kw)
        ref = orc.nuts(X, y, adapt_step_size=True, **kw)
        tol = _bar(orc, X, y, ref, adapt_step_size=True, **kw)
        np.testing.assert_allclose(r["step_size"][0], ref["step_size"], rtol=tol)
        np.testing.assert_allclose(r["inv_mass"][0], ref["inv_mass"], rtol=tol)
        compare_chain(r["samples"][0], r["stats"][0], ref, atol=tol)


def test_adaptation_many_chains_per_chain_data(sampler, orc):
    # one wave per chain, every chain its own data set and its own step size
    wl = workloads.WORKLOADS["chains4096_n500_d9_f64"]
    chains = [0, 1, 2, 63, 64, 200]
    X, y = workloads.make_workload(wl, chains=list(range(256)))
    say("adapt per-chain data, 256 chains")
    kw = dict(step_size=0.05, max_tree_depth=wl.max_tree_depth, num_warmup=120, num_samples=20,
              seed=wl.seed)
    r = sampler.sample(X, y, num_chains=256, per_chain=True, adapt_step_size=True,
                       adapt_diag_mass=True, **kw)
    for c in chains:
        ref = orc.nuts(X[c], y[c], chain=c, adapt_step_size=True, adapt_diag_mass=True, **kw)
        tol = _bar(orc, X[c], y[c], ref, chain=c, adapt_step_size=True, adapt_diag_mass=True, **kw)
        np.testing.assert_allclose(r["step_size"][c], ref["step_size"], rtol=tol)
        compare_chain(r["samples"][c], r["stats"][c], ref, atol=tol)
    assert len(set(np.round(r["step_size"], 12))) > 200  # every chain adapts on its own


def test_adaptation_batch_path(sampler, orc):
    # fp32 shared data on the matrix-core path, 130 chains (two tiles)
    X, y, _ = workloads.make_logistic(3000, 20, w_scale=0.3, key=[73, 1], dtype="f32")
    say("adapt batch path", 3000, 20, 130)
    d = sampler.data(X, y)
    kw = dict(step_size=0.5, max_tree_depth=6, num_warmup=8, num_samples=3, seed=4)
    r = d.sample(num_chains=130, path=3, adapt_step_size=True, **kw)
    for c in (0, 1, 127, 128, 129):
        ref = orc.nuts(X.astype(np.float64), y, chain=c, adapt_step_size=True, **kw)
        np.testing.assert_allclose(r["step_size"][c], ref["step_size"], rtol=2e-4)
        st = r["stats"][c]
        for f in DECISION_FIELDS:
            assert np.array_equal(st[f], ref["stats"][f]), (c, f)
        np.testing.assert_allclose(r["samples"][c], ref["samples"], rtol=2e-4, atol=2e-4)


def test_target_accept_checked(sampler):
    import paper_1912_11554_amd as nuts
    X, y, _ = workloads.make_logistic(100, 3, w_scale=1.0, key=[62, 2])
    for bad in (1.0, 1.5, -0.2):
        with pytest.raises(nuts.NutsError) as e:
            sampler.sample(X, y, step_size=0.1, max_tree_depth=5, num_warmup=5, num_samples=2,
                           adapt_step_size=True, target_accept=bad)
        assert e.value.code == nuts.NUTS_EINVAL
