"""Exact pins for the oracle's diagonal-mass rules (readings R13 and R19).

The regularisation var' = (n / (n + 5)) var + 1e-3 * 5 / (n + 5) is the Stan
reference manual's convention, not a quantity the mathematics fixes, and its
statistical consequences cannot tell it from nearby constants: the window's
sample variance of autocorrelated NUTS states is not the target variance in
expectation (on a one-dimensional Gaussian at n = 30 it averaged 0.885 of
it).  So these tests recompute the rule from the very states the oracle
used: the states after each warmup iteration come from the oracle's trace
hook (R19) or from the same chain run without adaptation (R13, whose warmup
is an ordinary fixed-step run), their variance from numpy's two-pass
np.var(ddof=1), and the published constants.  A wrong window, denominator,
shrinkage weight, constant or normalisation fails exactly.
"""
import numpy as np
import pytest

import workloads


def _shrink(states):
    n = states.shape[0]
    var = np.var(states, axis=0, ddof=1)
    return (n / (n + 5.0)) * var + 1e-3 * (5.0 / (n + 5.0))


@pytest.mark.parametrize("W", [40, 41, 120])
def test_r13_mass_from_the_second_half_of_warmup(orc, W):
    X, y, _ = workloads.make_logistic(300, 5, w_scale=1.0, key=[91, W])
    kw = dict(step_size=0.05, max_tree_depth=8, seed=4)
    r = orc.nuts(X, y, num_warmup=W, num_samples=15, adapt_diag_mass=True, **kw)
    # the warmup of reading R13 is the fixed-step run with the identity mass
    plain = orc.nuts(X, y, num_warmup=0, num_samples=W, **kw)
    im = _shrink(plain["samples"][W // 2:])
    im = im / im.mean()
    np.testing.assert_allclose(r["inv_mass"], im, rtol=1e-12)
    # from iteration W on the chain runs with that inverse mass: the same
    # as resuming the plain run's state with it
    cont = orc.nuts(X, y, num_warmup=0, num_samples=15, init_q=plain["final_q"], first_iter=W,
                    inv_mass=im, **kw)
    for f in ("tree_depth", "num_steps", "proposal_index", "term_leaf", "direction_bits"):
        assert np.array_equal(r["stats"][f], cont["stats"][f]), f
    np.testing.assert_allclose(r["samples"], cont["samples"], rtol=1e-10, atol=1e-12)


def test_r13_trace_hook_is_the_plain_run(orc):
    # the trace hook records exactly the states the chain visited
    X, y, _ = workloads.make_logistic(200, 4, w_scale=1.0, key=92)
    kw = dict(step_size=0.05, max_tree_depth=8, seed=6)
    r = orc.nuts(X, y, num_warmup=30, num_samples=2, adapt_diag_mass=True, warmup_trace=True, **kw)
    plain = orc.nuts(X, y, num_warmup=0, num_samples=30, **kw)
    assert np.array_equal(r["warmup_q"], plain["samples"])
    assert np.all(r["warmup_eps"] == 0.05)


@pytest.mark.parametrize("W", [100, 260])
def test_r19_mass_is_the_last_windows_shrunk_variance(orc, W):
    # windowed adaptation with the step size: at the end of warmup the
    # inverse mass is the last slow window's shrunk variance, not normalised
    X, y, _ = workloads.make_logistic(400, 6, w_scale=1.0, key=[93, W])
    r = orc.nuts(X, y, step_size=0.05, max_tree_depth=8, num_warmup=W, num_samples=3, seed=8,
                 adapt_diag_mass=True, adapt_step_size=True, warmup_trace=True)
    wins = orc.mass_windows(W)
    a, b = wins[-1]
    assert b <= W
    np.testing.assert_allclose(r["inv_mass"], _shrink(r["warmup_q"][a:b]), rtol=1e-12)
    # the first window ends with its own variance in place: the step-size
    # heuristic restarts there, so the step changes right after it
    if len(wins) > 1:
        e0 = r["warmup_eps"]
        assert e0[wins[0][1]] != e0[wins[0][1] - 1]


def test_r19_one_dimensional_constant_dominates(orc):
    # a one-dimensional N(0, 1e-4) posterior (prior only, prior scale 0.01):
    # the variance term is below the regularisation, so a wrong constant or
    # weight is far outside the exact recomputation
    X = np.zeros((1, 1))
    y = np.zeros(1, np.uint8)
    W = 40
    (a, b), = orc.mass_windows(W)
    n = b - a
    for c in range(20):
        q0 = np.random.default_rng(c).normal(0.0, 0.01, 1)
        r = orc.nuts(X, y, step_size=0.01, max_tree_depth=10, num_warmup=W, num_samples=1, seed=3,
                     chain=c, prior_scale=0.01, adapt_diag_mass=True, adapt_step_size=True,
                     init_q=q0, warmup_trace=True)
        want = _shrink(r["warmup_q"][a:b])
        np.testing.assert_allclose(r["inv_mass"], want, rtol=1e-12)
        assert want[0] > 1e-3 * 5.0 / (n + 5.0)
