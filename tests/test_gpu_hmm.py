"""GPU parity of the semi-supervised HMM target (nuts_hmm_potential_grad,
nuts_hmm_sample) against the oracle.

Bars.  Both sides run fp64, but the device splits the unobserved steps over
64 lanes (segment products, prefix and suffix products over lanes, then a
re-run of each segment), so its roundings differ from the oracle's
sequential recursion.  Each scaled step is a few roundings; log p is a sum
of at most 512 logs of normalisers in (0, 1], and the expected counts are
sums of at most 512 probabilities: absolute errors stay near 1e-13, so U is
held to 1e-10 relative to max(1, |U|) and every gradient component to
1e-9 absolute.  Sampling: tree decisions bit-exact, positions, energies and
accept statistics within 1e-9 (the bar of the other fp64 paths); with
warmup step-size adaptation, within a bar the oracle sets for itself
(_adapt_bar).
"""
import numpy as np
import pytest

import workloads
from tests.gpu_common import compare_chain, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sampler():
    import paper_1912_11554_amd as nuts
    return nuts.Sampler(0)


def _seq(T, Tsup, K, V, key):
    w, z, _, _ = workloads.make_hmm(T=T, Tsup=Tsup, K=K, V=V, key=key)
    return w, z


def _check_potential(sampler, orc, w, z, K, V, Q):
    U, g = sampler.hmm_potential_grad(w, z, K, V, Q)
    for i in range(Q.shape[0]):
        ru, rg = orc.hmm_potential_grad(w, z, K, V, Q[i])
        assert abs(U[i] - ru) <= 1e-10 * max(1.0, abs(ru)), (i, U[i], ru)
        np.testing.assert_allclose(g[i], rg, rtol=0, atol=1e-9)
    return U, g


@pytest.mark.parametrize("T,Tsup,K,V", [
    (600, 100, 3, 10),   # the paper's shape: 500 unobserved steps, 8 per lane
    (612, 100, 3, 10),   # 512 unobserved steps: every lane full
    (1, 0, 2, 2),        # one step, nothing observed (uniform start, no transition)
    (50, 50, 3, 5),      # everything observed: no forward pass
    (51, 50, 3, 5),      # one unobserved step
    (64, 0, 4, 12),      # 64 steps, one per lane; K*K + K*V = 64 entry lanes
    (165, 100, 2, 30),   # 65 steps: two per lane on 33 lanes; 64 entry lanes
    (300, 1, 4, 3),      # a single observed state
])
def test_potential_matches_oracle(sampler, orc, T, Tsup, K, V):
    w, z = _seq(T, Tsup, K, V, key=[7, T * 100 + Tsup])
    D = orc.hmm_dim(K, V)
    rng = np.random.default_rng([8, T, K, V])
    # zero, moderate and large logits (at scale 30 emission probabilities
    # reach ~1e-26: the segment products lean on their rescaling)
    Q = np.concatenate([np.zeros((1, D)), rng.normal(0.0, 1.0, (5, D)), rng.normal(0.0, 6.0, (2, D)),
                        rng.normal(0.0, 30.0, (2, D))])
    say("hmm potential", T, Tsup, K, V)
    _check_potential(sampler, orc, w, z, K, V, Q)


def test_potential_many_points(sampler, orc):
    # 1000 positions (250 groups of four waves), nine checked one by one
    w, z = _seq(600, 100, 3, 10, key=6)
    Q = np.random.default_rng(9).normal(0.0, 1.5, (1000, 33))
    say("hmm potential 1000 points")
    import paper_1912_11554_amd as nuts
    U, g = sampler.hmm_potential_grad(w, z, 3, 10, Q)
    for i in (0, 1, 3, 4, 255, 256, 511, 998, 999):
        ru, rg = orc.hmm_potential_grad(w, z, 3, 10, Q[i])
        assert abs(U[i] - ru) <= 1e-10 * max(1.0, abs(ru))
        np.testing.assert_allclose(g[i], rg, rtol=0, atol=1e-9)
    assert nuts.hmm_dim(3, 10) == 33


def _adapt_bar(orc, hm, ref, **kw):
    """max(1e-9, 100 s), s the oracle's own largest relative change (step
    size, samples) when every element of the unit inverse mass moves by one
    ulp in a random direction, over two such draws: the warmup's dual
    averaging feeds last-bit differences of the accept statistics back into
    the step size, and the trajectories amplify them (as for the logistic
    target's adaptation bar)."""
    rng = np.random.default_rng(4321)
    D = orc.hmm_dim(hm["K"], hm["V"])
    s = 0.0
    for _ in range(2):
        im = np.nextafter(np.ones(D), rng.choice([-np.inf, np.inf], size=D))
        b = orc.nuts(None, None, hmm=hm, inv_mass=im, **kw)
        s = max(s, abs(b["step_size"] / ref["step_size"] - 1.0),
                np.max(np.abs(b["samples"] - ref["samples"]) / (1.0 + np.abs(ref["samples"]))))
    return max(1e-9, 100.0 * s)


@pytest.mark.parametrize("adapt", [False, True])
def test_sampler_matches_oracle(sampler, orc, adapt):
    w, z = _seq(600, 100, 3, 10, key=6)
    hm = dict(w=w, z=z, K=3, V=10)
    say("hmm sample paper shape adapt", adapt)
    kw = dict(step_size=0.1, max_tree_depth=8, num_warmup=30 if adapt else 5, num_samples=30,
              seed=11, adapt_step_size=adapt)
    r = sampler.hmm_sample(w, z, 3, 10, **kw)
    ref = orc.nuts(None, None, hmm=hm, **kw)
    tol = _adapt_bar(orc, hm, ref, **kw) if adapt else 1e-9
    compare_chain(r["samples"][0], r["stats"][0], ref, atol=tol)
    assert r["grad_evals"] == ref["grad_evals"]
    if adapt:
        np.testing.assert_allclose(r["step_size"][0], ref["step_size"], rtol=tol)
        assert ref["step_size"] != 0.1


def test_sampler_many_chains(sampler, orc):
    # 300 chains (75 groups), inverse mass, the generalised criterion
    w, z = _seq(600, 100, 3, 10, key=6)
    hm = dict(w=w, z=z, K=3, V=10)
    im = np.linspace(0.5, 2.0, 33)
    kw = dict(step_size=0.08, max_tree_depth=7, num_warmup=3, num_samples=12, seed=5, inv_mass=im,
              uturn_generalized=True)
    say("hmm sample 300 chains")
    r = sampler.hmm_sample(w, z, 3, 10, num_chains=300, **kw)
    for c in (0, 1, 4, 150, 299):
        ref = orc.nuts(None, None, hmm=hm, chain=c, **kw)
        compare_chain(r["samples"][c], r["stats"][c], ref)


@pytest.mark.parametrize("T,Tsup,K,V", [(40, 0, 2, 4), (80, 79, 4, 6), (130, 10, 2, 9)])
def test_sampler_edge_shapes(sampler, orc, T, Tsup, K, V):
    w, z = _seq(T, Tsup, K, V, key=[12, T])
    hm = dict(w=w, z=z, K=K, V=V)
    say("hmm sample shape", T, Tsup, K, V)
    kw = dict(step_size=0.2, max_tree_depth=6, num_warmup=4, num_samples=15, seed=3,
              adapt_diag_mass=True)
    r = sampler.hmm_sample(w, z, K, V, **kw)
    ref = orc.nuts(None, None, hmm=hm, **kw)
    compare_chain(r["samples"][0], r["stats"][0], ref)


def test_rejects(sampler):
    import paper_1912_11554_amd as nuts
    w, z = _seq(100, 10, 3, 5, key=13)
    Q = np.zeros((1, 3 * 2 + 3 * 4))
    cases = [
        (dict(K=5, V=3), nuts.NUTS_EUNSUPPORTED),                 # K > 4
        (dict(K=4, V=13), nuts.NUTS_EUNSUPPORTED),                # 16 + 52 > 64 entries
        (dict(K=3, V=5, w=np.zeros(700, np.uint8)), nuts.NUTS_EUNSUPPORTED),  # 690 unobserved
        (dict(K=3, V=4, w=np.where(np.arange(100) == 7, 4, 0).astype(np.uint8)),
         nuts.NUTS_EINVAL),                                       # a symbol >= V
        (dict(K=3, V=5, z=np.full(10, 3, np.uint8)), nuts.NUTS_EINVAL),       # a state >= K
        (dict(K=3, V=5, z=np.zeros(200, np.uint8)), nuts.NUTS_EINVAL),        # Tsup > T
    ]
    for over, code in cases:
        a = dict(w=w, z=z, K=3, V=5)
        a.update(over)
        D = nuts.hmm_dim(a["K"], a["V"])
        with pytest.raises(nuts.NutsError) as e:
            sampler.hmm_potential_grad(a["w"], a["z"], a["K"], a["V"], np.zeros((1, D)))
        assert e.value.code == code, (over, e.value)
    with pytest.raises(nuts.NutsError) as e:
        sampler.hmm_sample(w, z, 3, 5, step_size=-1.0, max_tree_depth=5, num_warmup=0, num_samples=1)
    assert e.value.code == nuts.NUTS_EINVAL
    U, g = sampler.hmm_potential_grad(w, z, 3, 5, Q)
    assert np.isfinite(U).all() and np.isfinite(g).all()


def test_sampler_bench_configuration(sampler, orc):
    # the timed configuration of bench.py's HMM line: 8192 chains (2048
    # groups), depth 10, with an inverse mass; five chains checked over a
    # few iterations
    w, z = _seq(600, 100, 3, 10, key=6)
    hm = dict(w=w, z=z, K=3, V=10)
    im = np.linspace(0.6, 1.4, 33)
    kw = dict(step_size=0.15, max_tree_depth=10, num_warmup=2, num_samples=4, seed=2, inv_mass=im)
    say("hmm sample 8192 chains")
    r = sampler.hmm_sample(w, z, 3, 10, num_chains=8192, **kw)
    for c in (0, 1, 4095, 4096, 8191):
        ref = orc.nuts(None, None, hmm=hm, chain=c, **kw)
        compare_chain(r["samples"][c], r["stats"][c], ref)
