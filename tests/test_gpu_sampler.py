"""GPU parity of the device-resident NUTS against the oracle on identical
seeded inputs and identical Philox draws.

Bar (fp64): tree depth, step count, proposal index, termination leaf and
reason, direction bits bit-exact; positions, energies and acceptance
statistics within 1e-9 (the two sides sum in different orders).  fp32 X:
the same against the oracle on the fp32-rounded X promoted to fp64.
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


def _oracle_chain(orc, X, y, wl, chain, iters, **kw):
    return orc.nuts(X.astype(np.float64), y, step_size=wl.step_size,
                    max_tree_depth=wl.max_tree_depth, num_warmup=0, num_samples=iters,
                    seed=wl.seed, chain=chain, **kw)


@pytest.mark.parametrize("path", [1, 2])
def test_small_single_chain_50_iterations(sampler, orc, path):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("sampler logreg_n1000_d11 path", path)
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=50, seed=wl.seed, path=path)
    ref = _oracle_chain(orc, X, y, wl, 0, 50)
    compare_chain(r["samples"][0], r["stats"][0], ref)
    assert r["grad_evals"] == ref["grad_evals"]


def test_small_single_chain_full_run(sampler, orc):
    # the whole 200 + 200 run: warmup is not emitted, kept draws line up
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("sampler logreg_n1000_d11 full")
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=wl.num_warmup, num_samples=wl.num_samples, seed=wl.seed)
    ref = orc.nuts(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                   num_warmup=wl.num_warmup, num_samples=wl.num_samples, seed=wl.seed)
    compare_chain(r["samples"][0], r["stats"][0], ref)
    np.testing.assert_allclose(r["final_q"][0], ref["final_q"], rtol=1e-9, atol=1e-9)


@pytest.mark.parametrize("path", [1, 2])
def test_edge_cases_tiny(sampler, orc, path):
    # N = 1, D = 1; N = 65 (ragged block); forced divergence; max depth 1
    cases = [(1, 1, 0.5, 5), (65, 3, 0.2, 6), (200, 4, 5.0, 6), (100, 2, 0.01, 1),
             (130, 63, 0.05, 4)]
    for N, D, eps, maxd in cases:
        X, y, _ = workloads.make_logistic(N, D, w_scale=1.0, key=[60, N * 1000 + D])
        say("sampler tiny", N, D, eps, maxd, "path", path)
        r = sampler.sample(X, y, step_size=eps, max_tree_depth=maxd, num_warmup=3,
                           num_samples=20, seed=9, path=path)
        ref = orc.nuts(X, y, step_size=eps, max_tree_depth=maxd, num_warmup=3,
                       num_samples=20, seed=9)
        compare_chain(r["samples"][0], r["stats"][0], ref)


@pytest.mark.parametrize("D,path", [(64, 1), (64, 2), (129, 2), (257, 2)])
def test_wide_models(sampler, orc, D, path):
    # several lanes per row and several dimensions per lane
    N = 3000
    X, y, _ = workloads.make_logistic(N, D, w_scale=0.1, key=[61, D])
    say("sampler wide", N, D, "path", path)
    r = sampler.sample(X, y, step_size=0.02, max_tree_depth=6, num_warmup=2, num_samples=8, seed=5,
                       path=path)
    ref = orc.nuts(X, y, step_size=0.02, max_tree_depth=6, num_warmup=2, num_samples=8, seed=5)
    compare_chain(r["samples"][0], r["stats"][0], ref)


@pytest.mark.parametrize("D", [16, 17])
@pytest.mark.parametrize("path", [1, 2])
def test_tree_sums_either_side_of_one_row(sampler, orc, D, path):
    # with D <= 16 the tree's sums over dimensions take the first 16 lanes
    # only; D = 16 and D = 17 sit either side of that switch
    N = 400
    X, y, _ = workloads.make_logistic(N, D, w_scale=0.5, key=[62, D])
    say("sampler one-row boundary", N, D, "path", path)
    r = sampler.sample(X, y, step_size=0.05, max_tree_depth=6, num_warmup=2, num_samples=10, seed=11,
                       path=path)
    ref = orc.nuts(X, y, step_size=0.05, max_tree_depth=6, num_warmup=2, num_samples=10, seed=11)
    compare_chain(r["samples"][0], r["stats"][0], ref)


def test_many_chains_per_chain_data_subset(sampler, orc):
    # 256 chains of the 4096-chain workload (own data per chain); every chain
    # compared with the oracle for its first 50 iterations
    wl = workloads.WORKLOADS["chains4096_n500_d9_f64"]
    C = 256
    X, y = workloads.make_workload(wl, chains=range(C))
    say("sampler per-chain C=256")
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=50, num_chains=C, seed=wl.seed,
                       per_chain=True)
    for c in range(0, C, 8):
        ref = _oracle_chain(orc, X[c], y[c], wl, c, 50)
        compare_chain(r["samples"][c], r["stats"][c], ref)


def test_many_chains_all_4096_first_iterations(sampler, orc):
    # the whole 4,096-chain workload (own 500 x 9 fp64 data set per chain) in
    # the launch the benchmark times (LDS-resident data, four chains a
    # group): every chain compared with the oracle for its first 5 iterations
    wl = workloads.WORKLOADS["chains4096_n500_d9_f64"]
    X, y = workloads.make_workload(wl)
    C, iters = X.shape[0], 5
    assert C == 4096
    say("sampler per-chain C=4096, first iterations")
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=iters, num_chains=C, seed=wl.seed, per_chain=True)
    for c in range(C):
        ref = _oracle_chain(orc, X[c], y[c], wl, c, iters)
        compare_chain(r["samples"][c], r["stats"][c], ref)
    assert r["grad_evals"] == sum(int(r["stats"][c]["num_steps"].sum()) + 1 for c in range(C))


def test_shared_data_many_chains(sampler, orc):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("sampler shared data C=6")
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=30, num_chains=6, seed=3)
    for c in range(6):
        ref = orc.nuts(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=30, seed=3, chain=c)
        compare_chain(r["samples"][c], r["stats"][c], ref)


@pytest.mark.parametrize("path", [1, 2])
def test_resume_and_inv_mass(sampler, orc, path):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    im = np.linspace(0.5, 2.0, wl.D)
    q0 = np.full((1, wl.D), 0.1)
    say("sampler resume path", path)
    r = sampler.sample(X, y, step_size=0.04, max_tree_depth=8, num_warmup=0, num_samples=25,
                       seed=4, inv_mass=im, init_q=q0, first_iter=17, path=path)
    ref = orc.nuts(X, y, step_size=0.04, max_tree_depth=8, num_warmup=0, num_samples=25, seed=4,
                   inv_mass=im, init_q=q0[0], first_iter=17)
    compare_chain(r["samples"][0], r["stats"][0], ref)


def test_diag_mass_adaptation(sampler, orc):
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("sampler adapt diag mass")
    r = sampler.sample(X, y, step_size=0.05, max_tree_depth=8, num_warmup=60, num_samples=20,
                       seed=2, adapt_diag_mass=True)
    ref = orc.nuts(X, y, step_size=0.05, max_tree_depth=8, num_warmup=60, num_samples=20,
                   seed=2, adapt_diag_mass=True)
    np.testing.assert_allclose(r["inv_mass"][0], ref["inv_mass"], rtol=1e-9)
    compare_chain(r["samples"][0], r["stats"][0], ref)


@pytest.mark.parametrize("name", ["covtype_n581012_d55_f64", "covtype_n581012_d55_f32"])
def test_covtype_first_iterations(sampler, orc, name):
    # full-size data, the grid path, the first iterations checked one by one
    wl = workloads.WORKLOADS[name]
    X, y = workloads.make_workload(wl)
    iters = 12
    say("sampler covtype grid", name, "iters", iters)
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=iters, seed=wl.seed, path=2)
    ref = _oracle_chain(orc, X, y, wl, 0, iters)
    # fp32 data: the per-row exp/log/reciprocal run in fp32 (~1e-6 relative
    # per row), so positions drift apart at the 1e-8 level over the run; the
    # acceptance statistic averages exp(-(H - H0)) over the leaves, and each
    # row's fp32-evaluated loss carries ~3e-8 absolute error, a random walk of
    # sqrt(2 N) 3e-8 = 3.2e-5 in H - H0 at N = 581,012: compared within 1.5e-4
    # (as in the 50-iteration test below)
    compare_chain(r["samples"][0], r["stats"][0], ref, atol=1e-9 if wl.dtype == "f64" else 1e-6,
                  accept_atol=None if wl.dtype == "f64" else 1.5e-4)


@pytest.mark.parametrize("name", ["covtype_n581012_d55_f64", "covtype_n581012_d55_f32"])
def test_covtype_50_iterations_from_generating_weights(sampler, orc, name):
    # the 581,012 x 55 workload on the grid path in the benchmark's launch
    # shape, 50 iterations from the generating weights (in the posterior's
    # bulk: trees of typical length), every decision and position checked
    wl = workloads.WORKLOADS[name]
    X, y = workloads.make_workload(wl)
    _, _, w_true = workloads.make_logistic(1, wl.D, w_scale=wl.w_scale, key=wl.data_seed)
    iters = 50
    say("sampler covtype grid from w_true", name, "iters", iters)
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=iters, seed=wl.seed, path=2, init_q=w_true)
    ref = _oracle_chain(orc, X, y, wl, 0, iters, init_q=w_true)
    # The acceptance statistic averages exp(-(H - H0)) over the leaves, an
    # absolute quantity from the difference of two energies of ~5e4.  fp64:
    # the two sides' energies agree to ~1e-13 of their size (summation order,
    # carried along 50 iterations of trajectories), so it is compared within
    # 1e-12 |H|.  fp32: each row's loss is evaluated in fp32 (~3e-8 absolute
    # error), so H - H0 carries a random walk of sqrt(2 N) 3e-8 = 3.2e-5 at
    # N = 581,012; compared within 1.5e-4 (about 4.5 of those).
    H = np.abs(ref["stats"]["energy"]).max()
    n = compare_chain(r["samples"][0], r["stats"][0], ref,
                      atol=1e-9 if wl.dtype == "f64" else 1e-6,
                      accept_atol=1e-12 * H if wl.dtype == "f64" else 1.5e-4)
    assert n == iters
    assert r["grad_evals"] == ref["grad_evals"]


def test_streaming_workload_first_iterations(sampler, orc):
    # the 4,000,000 x 257 fp32 set (10 % of the features zero) on the grid
    # path in the launch shape the benchmark times (32-lane rows, 10 column
    # slots, lane-masked last slots, two block register sets), two
    # iterations from the generating weights checked one by one against the
    # oracle, which promotes the rows to fp64
    wl = workloads.WORKLOADS["stream_n4m_d257_f32"]
    X, y = workloads.make_workload(wl)
    _, _, w_true = workloads.make_logistic(1, wl.D, w_scale=wl.w_scale, key=wl.data_seed)
    iters = 2
    say("sampler 4M x 257 grid", "iters", iters)
    r = sampler.sample(X, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                       num_warmup=0, num_samples=iters, seed=wl.seed, path=2, init_q=w_true)
    X64 = X.astype(np.float64)
    ref = orc.nuts(X64, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                   num_warmup=0, num_samples=iters, seed=wl.seed, init_q=w_true)
    assert ref["stats"]["num_steps"].sum() >= 4  # real trees, not a divergence at the first leaf
    # the acceptance statistic averages exp(-(H - H0)) over the leaves, and
    # H - H0 is the difference of two 4,000,000-row sums whose row terms use
    # fp32 exp/log (about 6e-8 relative error per row, loss about 0.5 per
    # row): as a random walk that is sqrt(N) x 3e-8 = 6e-5 absolute in
    # H - H0, so the statistic is compared within 2e-4 (the energies
    # themselves, about 2e6, within 1e-6 relative)
    compare_chain(r["samples"][0], r["stats"][0], ref, atol=1e-6, accept_atol=2e-4)
    # the workload's diagonal mass (reading R13) across the end of warmup:
    # 4 warmup iterations (the mass from the states after iterations 2 and 3),
    # then 2 with it; depth 3 keeps the oracle's share to about 40 full
    # evaluations of the 4,000,000 rows
    say("sampler 4M x 257 grid, diagonal mass across the end of warmup")
    kw = dict(step_size=wl.step_size, max_tree_depth=3, num_warmup=4, num_samples=2,
              seed=wl.seed, init_q=w_true, adapt_diag_mass=True)
    r = sampler.sample(X, y, path=2, **kw)
    del X
    ref = orc.nuts(X64, y, **kw)
    np.testing.assert_allclose(r["inv_mass"][0], ref["inv_mass"], rtol=1e-5)
    # the rule's 1e-3 regularisation outweighs these states' variances
    # (~1e-6), so the normalised mass moves off one only slightly, but it moves
    assert np.abs(ref["inv_mass"] - 1.0).max() > 1e-6
    compare_chain(r["samples"][0], r["stats"][0], ref, atol=1e-6, accept_atol=2e-4)


@pytest.mark.parametrize("D", [65, 80, 128, 129, 160, 256, 257, 288, 289, 320])
def test_grid_fp32_wide_rows(sampler, orc, D):
    # fp32 data on the grid path, rows of 16 and 32 lanes: the loads of the
    # column slots past D - 1 are lane-masked and the streaming waves
    # alternate two block register sets; D at and around the slot
    # boundaries, a ragged last block
    N = 1237
    X, y, _ = workloads.make_logistic(N, D, w_scale=0.1, key=[67, D], dtype="f32")
    say("sampler grid fp32 wide", N, D)
    kw = dict(step_size=0.02, max_tree_depth=5, num_warmup=1, num_samples=4, seed=7)
    r = sampler.sample(X, y, path=2, **kw)
    ref = orc.nuts(X.astype(np.float64), y, **kw)
    # the acceptance statistic averages exp(-(H - H0)) over the leaves; each
    # row's fp32-evaluated loss carries about 3e-8 absolute error, so with no
    # cancellation between the two sums H - H0 is off by at most 3e-8 N
    compare_chain(r["samples"][0], r["stats"][0], ref, atol=1e-6, accept_atol=3e-8 * N)


@pytest.mark.parametrize("path", [1, 2])
def test_kernel_time_is_reported(sampler, path):
    # nuts_sample_opts.out_kernel_ms: events around the sampler kernel alone,
    # so positive and no longer than the whole call; the draws are the same
    # with and without the timing
    import time
    wl = workloads.WORKLOADS["logreg_n1000_d11_f64"]
    X, y = workloads.make_workload(wl)
    say("kernel time path", path)
    d = sampler.data(X, y)
    kw = dict(step_size=wl.step_size, max_tree_depth=wl.max_tree_depth, num_warmup=5, num_samples=20,
              seed=wl.seed, path=path)
    r0 = d.sample(**kw)
    t0 = time.perf_counter()
    r1 = d.sample(time_kernel=True, **kw)
    wall_ms = (time.perf_counter() - t0) * 1e3
    d.free()
    assert r0["kernel_ms"] is None
    assert 0.0 < r1["kernel_ms"] <= wall_ms
    np.testing.assert_array_equal(r0["samples"], r1["samples"])
    assert r0["grad_evals"] == r1["grad_evals"]


# Shapes of the grid path with enough row blocks that every worker keeps the
# last blocks of its share in LDS for the whole launch (the group's LDS
# beside the chain's state holds two or three of them a worker; each worker
# has at least four here, over 256 groups of 11 workers), and a ragged last
# block, which is one of the resident ones.  (D, dtype, rows per block,
# blocks a worker):
RESIDENT_SHAPES = [(9, "f32", 128, 4), (9, "f64", 128, 4), (20, "f32", 32, 5), (55, "f64", 8, 6),
                   (100, "f32", 8, 5), (150, "f64", 2, 5)]


@pytest.mark.parametrize("D,dt,R,per_wave", RESIDENT_SHAPES)
def test_grid_resident_blocks(sampler, orc, D, dt, R, per_wave):
    N = R * 256 * 11 * per_wave + R // 2 + 1
    X, y, w = workloads.make_logistic(N, D, w_scale=0.5, key=[75, D], dtype=dt)
    say("sampler grid resident blocks", N, D, dt)
    kw = dict(step_size=0.0015 * np.sqrt(581012 / N), max_tree_depth=6, num_warmup=1, num_samples=4,
              seed=13, init_q=w)
    r = sampler.sample(X, y, path=2, **kw)
    ref = orc.nuts(X.astype(np.float64), y, **kw)
    assert ref["stats"]["num_steps"].sum() >= 8  # trees, not divergences at the first leaf
    if dt == "f64":
        H = np.abs(ref["stats"]["energy"]).max()
        compare_chain(r["samples"][0], r["stats"][0], ref, atol=1e-9, accept_atol=1e-12 * H)
    else:
        # each row's fp32-evaluated loss carries about 3e-8 absolute error
        # (random in sign): H - H0 within 5 sqrt(2 N) 3e-8
        compare_chain(r["samples"][0], r["stats"][0], ref, atol=1e-6,
                      accept_atol=5 * np.sqrt(2 * N) * 3e-8)
    assert r["grad_evals"] == ref["grad_evals"]
