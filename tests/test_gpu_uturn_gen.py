"""GPU parity of the generalised U-turn criterion (NUTS_UTURN_GENERALIZED)
against the oracle, on every path.  Bars as for the endpoint criterion: fp64
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
def test_generalised_small_chain(sampler, orc, path):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("uturn generalised logreg path", path)
    kw = dict(step_size=wl.step_size, max_tree_depth=wl.max_tree_depth, num_warmup=10,
              num_samples=50, seed=wl.seed)
    r = sampler.sample(X, y, path=path, uturn_generalized=True, **kw)
    ref = orc.nuts(X, y, uturn_generalized=True, **kw)
    compare_chain(r["samples"][0], r["stats"][0], ref)
    assert r["grad_evals"] == ref["grad_evals"]
    # and it is not the endpoint criterion's run
    base = orc.nuts(X, y, **kw)
    assert not np.array_equal(base["stats"]["num_steps"], ref["stats"]["num_steps"])


@pytest.mark.parametrize("path", [1, 2])
def test_generalised_edge_cases(sampler, orc, path):
    cases = [(1, 1, 0.5, 5), (65, 3, 0.2, 6), (200, 4, 5.0, 6), (100, 2, 0.01, 1),
             (130, 63, 0.05, 4)]
    for N, D, eps, maxd in cases:
        X, y, _ = workloads.make_logistic(N, D, w_scale=1.0, key=[60, N * 1000 + D])
        say("uturn generalised tiny", N, D, eps, maxd, "path", path)
        kw = dict(step_size=eps, max_tree_depth=maxd, num_warmup=3, num_samples=20, seed=9,
                  inv_mass=np.linspace(0.5, 1.5, D))
        r = sampler.sample(X, y, path=path, uturn_generalized=True, **kw)
        ref = orc.nuts(X, y, uturn_generalized=True, **kw)
        compare_chain(r["samples"][0], r["stats"][0], ref)


@pytest.mark.parametrize("D", [129, 257])
def test_generalised_wide_grid(sampler, orc, D):
    N = 3000
    X, y, _ = workloads.make_logistic(N, D, w_scale=0.1, key=[61, D])
    say("uturn generalised wide", N, D)
    kw = dict(step_size=0.02, max_tree_depth=6, num_warmup=2, num_samples=8, seed=5)
    r = sampler.sample(X, y, path=2, uturn_generalized=True, **kw)
    ref = orc.nuts(X, y, uturn_generalized=True, **kw)
    compare_chain(r["samples"][0], r["stats"][0], ref)


def test_generalised_with_adaptation(sampler, orc):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("uturn generalised + adaptation")
    kw = dict(step_size=0.3, max_tree_depth=wl.max_tree_depth, num_warmup=60, num_samples=20,
              seed=wl.seed)
    r = sampler.sample(X, y, path=1, uturn_generalized=True, adapt_step_size=True, **kw)
    ref = orc.nuts(X, y, uturn_generalized=True, adapt_step_size=True, **kw)
    np.testing.assert_allclose(r["step_size"][0], ref["step_size"], rtol=1e-9)
    compare_chain(r["samples"][0], r["stats"][0], ref, atol=1e-8)


def test_generalised_batch_path(sampler, orc):
    X, y, _ = workloads.make_logistic(500, 129, w_scale=0.3, key=[72, 500 * 1000 + 129], dtype="f32")
    say("uturn generalised batch", 500, 129, 24)
    d = sampler.data(X, y)
    kw = dict(step_size=0.02, max_tree_depth=6, num_warmup=1, num_samples=5, seed=9)
    r = d.sample(num_chains=24, path=3, uturn_generalized=True, **kw)
    for c in (0, 7, 23):
        ref = orc.nuts(X.astype(np.float64), y, chain=c, uturn_generalized=True, **kw)
        st = r["stats"][c]
        for f in DECISION_FIELDS:
            assert np.array_equal(st[f], ref["stats"][f]), (c, f)
        np.testing.assert_allclose(r["samples"][c], ref["samples"], rtol=1e-5, atol=1e-5)
