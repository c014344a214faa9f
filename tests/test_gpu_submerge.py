"""GPU parity of merge-structured subtree proposals (NUTS_SUBTREE_MERGE)
against the oracle, on every path.  Bars as for the streaming choice: fp64
decisions bit-exact, positions, energies and accept statistics within 1e-9;
fp32 data on the matrix-core path: decisions bit-exact, positions within
1e-5."""
import numpy as np
import pytest

import workloads
from tests.gpu_common import DECISION_FIELDS, compare_chain, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sampler():
    import paper_1912_11554_amd as nuts
    return nuts.Sampler(0)


@pytest.mark.parametrize("path", [1, 2])
def test_submerge_small_chain(sampler, orc, path):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("subtree merge logreg path", path)
    kw = dict(step_size=wl.step_size, max_tree_depth=wl.max_tree_depth, num_warmup=10,
              num_samples=50, seed=wl.seed)
    r = sampler.sample(X, y, path=path, subtree_merge=True, **kw)
    ref = orc.nuts(X, y, subtree_merge=True, **kw)
    compare_chain(r["samples"][0], r["stats"][0], ref)
    assert r["grad_evals"] == ref["grad_evals"]
    base = orc.nuts(X, y, **kw)
    assert not np.array_equal(base["stats"]["proposal_index"], ref["stats"]["proposal_index"])


@pytest.mark.parametrize("path", [1, 2])
def test_submerge_edge_cases(sampler, orc, path):
    cases = [(1, 1, 0.5, 5), (65, 3, 0.2, 6), (200, 4, 5.0, 6), (100, 2, 0.01, 1),
             (130, 63, 0.05, 4)]
    for N, D, eps, maxd in cases:
        X, y, _ = workloads.make_logistic(N, D, w_scale=1.0, key=[63, N * 1000 + D])
        say("subtree merge tiny", N, D, eps, maxd, "path", path)
        kw = dict(step_size=eps, max_tree_depth=maxd, num_warmup=3, num_samples=20, seed=9,
                  inv_mass=np.linspace(0.5, 1.5, D))
        r = sampler.sample(X, y, path=path, subtree_merge=True, **kw)
        ref = orc.nuts(X, y, subtree_merge=True, **kw)
        compare_chain(r["samples"][0], r["stats"][0], ref)


@pytest.mark.parametrize("D", [129, 257])
def test_submerge_wide_grid(sampler, orc, D):
    X, y, _ = workloads.make_logistic(3000, D, w_scale=0.1, key=[64, D])
    say("subtree merge wide", D)
    kw = dict(step_size=0.02, max_tree_depth=6, num_warmup=2, num_samples=8, seed=5)
    r = sampler.sample(X, y, path=2, subtree_merge=True, **kw)
    ref = orc.nuts(X, y, subtree_merge=True, **kw)
    compare_chain(r["samples"][0], r["stats"][0], ref)


def test_submerge_with_other_features(sampler, orc):
    # with the generalised criterion and warmup adaptation (fixed-step bar
    # for the criterion; adaptation with the self-calibrated bar of the
    # adaptation tests would be looser, so the step size is held here)
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("subtree merge + generalised criterion")
    kw = dict(step_size=0.1, max_tree_depth=8, num_warmup=5, num_samples=40, seed=3,
              uturn_generalized=True)
    for path in (1, 2):
        r = sampler.sample(X, y, path=path, subtree_merge=True, **kw)
        ref = orc.nuts(X, y, subtree_merge=True, **kw)
        compare_chain(r["samples"][0], r["stats"][0], ref)
    say("subtree merge + adaptation")
    kw = dict(step_size=0.3, max_tree_depth=8, num_warmup=40, num_samples=10, seed=3,
              adapt_step_size=True)
    r = sampler.sample(X, y, path=1, subtree_merge=True, **kw)
    ref = orc.nuts(X, y, subtree_merge=True, **kw)
    for f in DECISION_FIELDS:
        assert np.array_equal(r["stats"][0][f], ref["stats"][f]), f
    np.testing.assert_allclose(r["step_size"][0], ref["step_size"], rtol=1e-6)


def test_submerge_many_chains_deep_tree(sampler, orc):
    # per-chain data, 64 chains; then depth 30 with D = 64, whose tree state
    # (S and the merge stack, 77.5 KB per chain) leaves room for two chains
    # per group on the streaming (non-resident) variant
    wl = workloads.WORKLOADS["chains4096_n500_d9_f64"]
    X, y = workloads.make_workload(wl, chains=list(range(64)))
    say("subtree merge per-chain data, 64 chains")
    kw = dict(step_size=wl.step_size, max_tree_depth=wl.max_tree_depth, num_warmup=5,
              num_samples=20, seed=wl.seed)
    r = sampler.sample(X, y, num_chains=64, per_chain=True, subtree_merge=True, **kw)
    for c in (0, 33, 63):
        ref = orc.nuts(X[c], y[c], chain=c, subtree_merge=True, **kw)
        compare_chain(r["samples"][c], r["stats"][c], ref)
    X2, y2, _ = workloads.make_logistic(400, 64, w_scale=0.3, key=[65, 1])
    say("subtree merge depth 30, D 64, 3 chains")
    kw = dict(step_size=0.05, max_tree_depth=30, num_warmup=2, num_samples=6, seed=2)
    r = sampler.sample(X2, y2, num_chains=3, path=1, subtree_merge=True, **kw)
    for c in range(3):
        ref = orc.nuts(X2, y2, chain=c, subtree_merge=True, **kw)
        compare_chain(r["samples"][c], r["stats"][c], ref)


def test_submerge_batch_path(sampler, orc):
    X, y, _ = workloads.make_logistic(500, 129, w_scale=0.3, key=[74, 500 * 1000 + 129], dtype="f32")
    say("subtree merge batch", 500, 129, 24)
    d = sampler.data(X, y)
    kw = dict(step_size=0.02, max_tree_depth=6, num_warmup=1, num_samples=5, seed=9)
    r = d.sample(num_chains=24, path=3, subtree_merge=True, **kw)
    for c in (0, 7, 23):
        ref = orc.nuts(X.astype(np.float64), y, chain=c, subtree_merge=True, **kw)
        st = r["stats"][c]
        for f in DECISION_FIELDS:
            assert np.array_equal(st[f], ref["stats"][f]), (c, f)
        np.testing.assert_allclose(r["samples"][c], ref["samples"], rtol=1e-5, atol=1e-5)
    d.free()


def test_submerge_hmm(sampler, orc):
    w, z, _, _ = workloads.make_hmm(key=6)
    hm = dict(w=w, z=z, K=3, V=10)
    say("subtree merge hmm")
    kw = dict(step_size=0.1, max_tree_depth=8, num_warmup=5, num_samples=25, seed=11)
    r = sampler.hmm_sample(w, z, 3, 10, num_chains=2, subtree_merge=True, **kw)
    for c in range(2):
        ref = orc.nuts(None, None, hmm=hm, chain=c, subtree_merge=True, **kw)
        compare_chain(r["samples"][c], r["stats"][c], ref)


def test_grid_tree_state_too_large(sampler):
    import paper_1912_11554_amd as nuts
    X, y, _ = workloads.make_logistic(2000, 257, w_scale=0.1, key=[66, 1])
    with pytest.raises(nuts.NutsError) as e:
        sampler.sample(X, y, path=2, step_size=0.01, max_tree_depth=30, num_warmup=0,
                       num_samples=1, subtree_merge=True)
    assert e.value.code == nuts.NUTS_EUNSUPPORTED
