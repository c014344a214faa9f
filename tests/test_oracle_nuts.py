"""Pins for the oracle's NUTS: recursive (Alg. 1) and iterative (Alg. 2)
builders give identical trees and proposals under the same draws; tree
bookkeeping invariants; resumability; and the sampled distribution matches
closed forms (conjugate Gaussian, prior-only, one-dimensional quadrature)
within 4 Monte Carlo standard errors."""
import numpy as np
import pytest
from scipy import integrate, optimize, special

import workloads
from oracle.ess import ess_columns


def _tiny(seed, N, D):
    X, y, _ = workloads.make_logistic(N, D, w_scale=1.5, key=[100, seed])
    return X, y


CASES = [
    # (step size, max depth): ordinary, divergent, saturating at max depth
    (0.3, 6),
    (0.8, 8),
    (6.0, 6),
    (1e-3, 5),
]


@pytest.mark.parametrize("eps,maxd", CASES)
def test_recursive_equals_iterative(orc, eps, maxd):
    seen = dict(div=0, turn_inside=0, turn_traj=0, maxd=0)
    for seed in range(40):
        N, D = 5 + seed % 16, 1 + seed % 3
        X, y = _tiny(seed, N, D)
        kw = dict(step_size=eps, max_tree_depth=maxd, num_warmup=5, num_samples=15,
                  seed=seed, chain=seed % 3, trace_cap=1 << 14,
                  inv_mass=np.linspace(0.5, 1.5, D))
        a = orc.nuts(X, y, builder=orc.BUILDER_ITERATIVE, **kw)
        b = orc.nuts(X, y, builder=orc.BUILDER_RECURSIVE, **kw)
        assert np.array_equal(a["samples"], b["samples"])
        assert a["stats"].tobytes() == b["stats"].tobytes()
        assert np.array_equal(a["trace"], b["trace"])
        assert a["grad_evals"] == b["grad_evals"]
        st = a["stats"]
        seen["div"] += int(st["diverging"].sum())
        seen["turn_inside"] += int(((st["term_leaf"] >= 0) & (st["turning"] == 1)).sum())
        seen["turn_traj"] += int((st["term_leaf"] == -2).sum())
        seen["maxd"] += int(st["hit_max_depth"].sum())
    # each case exercises the path it is meant for
    if eps >= 6.0:
        assert seen["div"] > 0
    elif eps <= 1e-3:
        assert seen["maxd"] > 0
    else:
        assert seen["turn_inside"] > 0 and seen["turn_traj"] > 0


def test_tree_bookkeeping_invariants(orc):
    X, y = _tiny(1, 40, 3)
    for eps, maxd in CASES:
        r = orc.nuts(X, y, step_size=eps, max_tree_depth=maxd, num_warmup=0, num_samples=300,
                     seed=3)
        st = r["stats"]
        d = st["tree_depth"].astype(np.int64)
        assert (d >= 1).all() and (d <= maxd).all()
        assert (st["direction_bits"] < (1 << d)).all()
        full = st["term_leaf"] < 0
        # a completed trajectory of depth d has 2^d - 1 leapfrog steps
        assert (st["num_steps"][full] == (1 << d[full]) - 1).all()
        # a subtree stopped at leaf n adds n + 1 steps to the earlier 2^(d-1) - 1
        part = ~full
        assert (st["num_steps"][part] == (1 << (d[part] - 1)) - 1 + st["term_leaf"][part] + 1).all()
        assert (np.abs(st["proposal_index"]) <= (1 << d) - 1).all()
        assert (st["hit_max_depth"] == ((d == maxd) & full & (st["turning"] == 0))).all()
        assert ((st["diverging"] == 1) <= part).all()
        assert (st["accept_prob"] >= 0).all() and (st["accept_prob"] <= 1).all()
        assert r["grad_evals"] == st["num_steps"].sum() + 1
        # the reported potential is U at the reported sample
        for k in range(0, 300, 37):
            U, _ = orc.logistic_potential_grad(X, y, r["samples"][k])
            assert st["potential_energy"][k] == U


def test_resume_is_exact(orc):
    X, y = _tiny(2, 30, 2)
    kw = dict(step_size=0.4, max_tree_depth=6, seed=8, chain=1)
    full = orc.nuts(X, y, num_warmup=0, num_samples=60, **kw)
    a = orc.nuts(X, y, num_warmup=0, num_samples=30, **kw)
    b = orc.nuts(X, y, num_warmup=0, num_samples=30, init_q=a["final_q"], first_iter=30, **kw)
    assert np.array_equal(full["samples"], np.concatenate([a["samples"], b["samples"]]))
    assert full["stats"].tobytes() == np.concatenate([a["stats"], b["stats"]]).tobytes()


def _within_mcse(samples, mean_true, var_true, k=4.0):
    """samples [C, n, D]: the mean and the second central moment each lie
    within k Monte Carlo standard errors of the truth."""
    flat = samples.reshape(-1, samples.shape[-1])
    ess_m = ess_columns(samples)
    mcse_m = flat.std(axis=0, ddof=1) / np.sqrt(ess_m)
    assert (np.abs(flat.mean(0) - mean_true) < k * mcse_m).all(), (flat.mean(0), mean_true,
                                                                    mcse_m)
    sq = (samples - mean_true) ** 2
    ess_v = ess_columns(sq)
    mcse_v = sq.reshape(-1, sq.shape[-1]).std(axis=0, ddof=1) / np.sqrt(ess_v)
    assert (np.abs(sq.reshape(-1, sq.shape[-1]).mean(0) - var_true) < k * mcse_v).all(), (
        sq.reshape(-1, sq.shape[-1]).mean(0), var_true, mcse_v)


def _run_chains(orc, X, y, C, **kw):
    return np.stack([orc.nuts(X, y, chain=c, **kw)["samples"] for c in range(C)])


@pytest.mark.slow
def test_conjugate_gaussian_posterior(orc):
    X, yv = workloads.make_lingauss(30, 3, key=21, noise_scale=0.5)
    s, sn = 2.0, 0.5
    P = X.T @ X / sn**2 + np.eye(3) / s**2
    Sigma = np.linalg.inv(P)
    mu = Sigma @ X.T @ yv / sn**2
    S = _run_chains(orc, X, None, 4, step_size=0.05, max_tree_depth=8, num_warmup=200,
                    num_samples=2000, seed=1, prior_scale=s, target=orc.TARGET_LINGAUSS,
                    yv=yv, noise_scale=sn)
    _within_mcse(S, mu, np.diag(Sigma))
    # off-diagonal covariance: sign and rough size
    emp = np.cov(S.reshape(-1, 3).T)
    np.testing.assert_allclose(emp, Sigma, atol=0.15 * np.sqrt(np.outer(np.diag(Sigma),
                                                                        np.diag(Sigma))).max())


@pytest.mark.slow
def test_prior_only_logistic(orc):
    # X = 0: the likelihood is constant, the posterior is N(0, s^2 I)
    s = 1.5
    X = np.zeros((5, 3))
    y = np.array([0, 1, 1, 0, 1], dtype=np.uint8)
    S = _run_chains(orc, X, y, 4, step_size=0.4, max_tree_depth=8, num_warmup=100,
                    num_samples=2000, seed=2, prior_scale=s)
    _within_mcse(S, np.zeros(3), np.full(3, s * s))


@pytest.mark.slow
def test_intercept_only_logistic_quadrature(orc):
    # D = 1 (the intercept column only): the posterior of b is one-dimensional
    X, y, _ = workloads.make_logistic(60, 1, w_scale=1.0, key=31)
    k, n = int(y.sum()), len(y)

    def logpost(b):
        return k * special.log_expit(b) + (n - k) * special.log_expit(-b) - 0.5 * b * b

    # adaptive quadrature around the mode, integrand scaled by its maximum
    mode = optimize.minimize_scalar(lambda b: -logpost(b)).x
    top = logpost(mode)
    dens = lambda b: np.exp(logpost(b) - top)
    lim = dict(a=mode - 8.0, b=mode + 8.0, points=[mode - 1, mode, mode + 1], limit=400)
    Z = integrate.quad(dens, **lim)[0]
    m1 = integrate.quad(lambda b: b * dens(b), **lim)[0] / Z
    m2 = integrate.quad(lambda b: (b - m1) ** 2 * dens(b), **lim)[0] / Z
    S = _run_chains(orc, X, y, 4, step_size=0.2, max_tree_depth=8, num_warmup=100,
                    num_samples=2500, seed=4)
    _within_mcse(S, np.array([m1]), np.array([m2]))


@pytest.mark.slow
def test_diag_mass_adaptation(orc):
    # strongly anisotropic Gaussian: after warmup the inverse mass follows the
    # posterior variances (mean-one normalised) and sampling stays exact
    sds = np.array([0.05, 1.0, 4.0])
    X = np.diag(1.0 / sds)           # one row per coordinate, unit noise
    yv = np.zeros(3)
    r = orc.nuts(X, None, step_size=0.02, max_tree_depth=10, num_warmup=400, num_samples=1500,
                 seed=5, prior_scale=1e6, target=orc.TARGET_LINGAUSS, yv=yv, noise_scale=1.0,
                 adapt_diag_mass=True)
    im = r["inv_mass"]
    assert im.mean() == pytest.approx(1.0, rel=1e-12)
    ratio = im / im[1]
    np.testing.assert_allclose(ratio[[0, 2]], (sds**2 / sds[1] ** 2)[[0, 2]], rtol=0.5)
    _within_mcse(r["samples"][None], np.zeros(3), sds**2)


def test_is_uturn_definition(orc):
    # Hoffman & Gelman: with left end (qL, pL) and right end (qR, pR) in time
    # order, the trajectory turns iff (qR - qL).M^-1 pL < 0 or
    # (qR - qL).M^-1 pR < 0; a zero dot product is not a turn.
    q0, q1 = np.array([0.0, 0.0]), np.array([1.0, 0.0])
    fwd, back, side = np.array([1.0, 0.0]), np.array([-1.0, 0.0]), np.array([0.0, 1.0])
    assert not orc.is_uturn(q0, fwd, q1, fwd, +1)
    assert orc.is_uturn(q0, fwd, q1, back, +1)          # right end turned back
    assert orc.is_uturn(q0, back, q1, fwd, +1)          # left end turned back
    assert not orc.is_uturn(q0, side, q1, side, +1)     # both dot products exactly 0
    # a subtree built backwards in time: first-generated node is the right end
    assert not orc.is_uturn(q1, fwd, q0, fwd, -1)
    assert orc.is_uturn(q0, fwd, q1, fwd, -1)
    # the inverse mass weights the momenta
    assert not orc.is_uturn(q0, np.array([1.0, 5.0]), q1 + np.array([0, 1.0]),
                            np.array([1.0, -2.0]), +1, inv_mass=np.array([1.0, 0.1]))
    assert orc.is_uturn(q0, np.array([1.0, 5.0]), q1 + np.array([0, 1.0]),
                        np.array([1.0, -2.0]), +1, inv_mass=np.array([1.0, 1.0]))


def _one_iteration(orc, X, y, q0, salt, **kw):
    return orc.nuts(X, y, num_warmup=0, num_samples=1, init_q=q0, first_iter=7, leaves_cap=4096,
                    sel_salt=salt, **kw)


# anisotropic 2-D Gaussian (sds 0.2 and 5): the stiff direction makes the leaf
# energies vary by O(1) while the soft one keeps the trajectory going
_SDS = np.array([0.2, 5.0])
_GAUSS = dict(target=1, yv=np.zeros(2), prior_scale=1e6, noise_scale=1.0)


def test_leaf_trace_energy_rules(orc):
    # divergence is flagged exactly at the first leaf whose H - H0 exceeds
    # Hoffman & Gelman's Delta_max = 1000; accept_prob is the leaf mean of
    # min(1, exp(-(H - H0))); leaf positions extend the trajectory by 2^j
    X, y = _tiny(6, 30, 2)
    n_div = n_mid = 0
    for eps in (0.3, 1.0, 1.5, 2.5, 4.0):
        for seed in range(30):
            r = orc.nuts(X, y, step_size=eps, max_tree_depth=7, num_warmup=0, num_samples=1,
                         seed=seed, leaves_cap=4096, init_q=np.array([0.3, -0.2]))
            st, lv = r["stats"][0], r["leaves"]
            dH = lv["dH"]
            n_mid += int(((dH > 1.0) & (dH <= 1000.0)).sum())
            big = np.flatnonzero(~(dH <= 1000.0))
            if st["diverging"]:
                n_div += 1
                assert len(big) == 1 and big[0] == len(dH) - 1
                assert lv["n"][-1] == st["term_leaf"]
            else:
                assert len(big) == 0
            acc = np.where(np.isnan(dH), 0.0, np.minimum(1.0, np.exp(-dH)))
            assert st["accept_prob"] == pytest.approx(acc.mean(), rel=1e-12)
            assert len(dH) == st["num_steps"]
            for j in np.unique(lv["j"]):
                pos = lv["pos"][lv["j"] == j]
                step = 1 if st["direction_bits"] >> j & 1 else -1
                assert (np.diff(pos) == step).all()
                assert abs(pos[0]) == (1 << j) if j == 0 else True
    # both sides of the threshold were exercised
    assert n_div > 0 and n_mid > 0


def test_proposal_index_reintegrates(orc):
    # the sample of an iteration is the leapfrog trajectory point at its
    # proposal index: |k| steps from the previous state in direction sign(k)
    X, y = _tiny(7, 25, 3)
    eps = 0.35
    r = orc.nuts(X, y, step_size=eps, max_tree_depth=6, num_warmup=0, num_samples=40, seed=12)
    prev = np.zeros(3)
    for t in range(40):
        k = int(r["stats"]["proposal_index"][t])
        p0 = orc.normals(12, 0, t, 3)
        q, _, _ = orc.leapfrog(X, y, prev, p0, eps if k >= 0 else -eps, abs(k))
        np.testing.assert_array_equal(q, r["samples"][t])
        prev = r["samples"][t]


def _exact_selection(leaves, st):
    """Exact probability of each trajectory position being the sample under
    multinomial selection inside each subtree and biased progressive
    selection min(1, W_subtree / W_trajectory) at each merge."""
    prob = {0: 1.0}
    W_traj = 1.0                      # the initial leaf has weight exp(0)
    last_ok = st["tree_depth"] - (1 if st["term_leaf"] >= 0 else 0)
    for j in range(last_ok):
        sel = leaves["j"] == j
        w = np.exp(-leaves["dH"][sel])
        W_sub = w.sum()
        a = min(1.0, W_sub / W_traj)
        prob = {k: (1 - a) * v for k, v in prob.items()}
        for pos, wi in zip(leaves["pos"][sel], w):
            prob[int(pos)] = prob.get(int(pos), 0.0) + a * wi / W_sub
        W_traj += W_sub
    return prob


@pytest.mark.slow
@pytest.mark.parametrize("eps,seed", [(0.3, 2), (0.35, 0)])
def test_selection_distribution(orc, eps, seed):
    # over a fixed trajectory, re-drawing only the selection uniforms must
    # reproduce the exact selection probabilities (chi-square test)
    from scipy import stats as sst
    X, y = np.diag(1.0 / _SDS), None
    q0 = np.array([0.1, 2.0])
    kw = dict(step_size=eps, max_tree_depth=6, seed=seed, **_GAUSS)
    ref = _one_iteration(orc, X, y, q0, 0, **kw)
    assert ref["leaves"]["dH"].max() - ref["leaves"]["dH"].min() > 0.5
    prob = _exact_selection(ref["leaves"], ref["stats"][0])
    counts = {}
    R = 20000
    for salt in range(1, R + 1):
        r = _one_iteration(orc, X, y, q0, salt, **kw)
        assert np.array_equal(r["leaves"]["dH"], ref["leaves"]["dH"])
        k = int(r["stats"]["proposal_index"][0])
        counts[k] = counts.get(k, 0) + 1
    assert set(counts) <= set(prob)
    keys = sorted(prob)
    obs = np.array([counts.get(k, 0) for k in keys], dtype=float)
    exp = np.array([prob[k] for k in keys]) * R
    assert len(keys) >= 4 and abs(sum(prob.values()) - 1) < 1e-12
    # merge sparse cells so every expected count is >= 5
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
