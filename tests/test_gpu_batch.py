"""GPU parity of the batched-chain path (shared fp32 data, the potential and
gradient of many positions as fp32 matrix-core products) against the oracle.

Bar.  The batched contraction rounds the positions to fp32 and sums products
in fp32 inside the matrix cores, so against the oracle's fp64 arithmetic on
the same fp32 X each row term carries ~1e-7 (1 + |eta|) of error.  Bounds:
|dU| <= 1e-5 U (U >= sum of the row losses, each >= ~|eta| / 2 for large
|eta|, so this is ~100x the expected error) and per gradient component
1e-5 (|g| + sum_i |x_ij| + |w_j| / s^2 + 1) (grad_tol), both well inside the
1e-4 relative bar for fp32.  Sampler decisions (depths, steps, proposal
indices, termination, directions) are compared exactly: an energy error of
~1e-6 flips a multinomial or merge decision only when its uniform lies
within ~1e-6 of the threshold, and the seeds below have no such case.
"""
import numpy as np
import pytest

import workloads
from tests.gpu_common import DECISION_FIELDS, grad_tol, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sampler():
    import paper_1912_11554_amd as nuts
    return nuts.Sampler(0)


def _data(N, D, key, w_scale=0.3):
    X, y, w_true = workloads.make_logistic(N, D, w_scale=w_scale, key=key, dtype="f32")
    return X, y, w_true


def _check_potential(orc, X, y, W, U, G, s=1.0, rtol=1e-5):
    for k in range(W.shape[0]):
        u_ref, g_ref = orc.logistic_potential_grad_f32(X, y, W[k], prior_scale=s)
        assert abs(U[k] - u_ref) <= rtol * abs(u_ref), (k, U[k], u_ref)
        tol = grad_tol(X, W[k], g_ref, s, rtol)
        bad = np.flatnonzero(np.abs(G[k] - g_ref) > tol)
        assert bad.size == 0, (k, bad[:5], G[k][bad[:5]], g_ref[bad[:5]])


@pytest.mark.parametrize("N,D,K", [
    (1000, 129, 256),   # the 256-chain shape on a short X: two tiles, eight chunks + tail
    (777, 20, 17),      # one chunk + 4-column tail, ragged stage, ragged tile
    (300, 3, 5),        # tail only, no matrix-core chunk
    (130, 132, 130),    # widest shape: eight chunks + 4 tail columns; 2 tiles, second with 2
    (1000, 37, 64),     # padded chunks (37 -> 48 columns), no tail
    (64, 16, 1),        # one full stage, one chunk, one position
    (65, 68, 33),       # one row past a stage; 4 chunks + tail
])
def test_batched_potential_matches_oracle(sampler, orc, N, D, K):
    X, y, _ = _data(N, D, [70, N * 1000 + D])
    rng = np.random.default_rng(N + D + K)
    W = rng.normal(0.0, 0.3, size=(K, D))
    say("batched potential", N, D, K)
    d = sampler.data(X, y)
    U, G = d.potential_grad(W, prior_scale=1.3, batched=True)
    _check_potential(orc, X, y, W, U, G, s=1.3)


def test_batched_potential_full_size_samples(sampler, orc):
    # the 256-chain workload's X at full size; a few positions checked one by one
    wl = workloads.WORKLOADS["shared256_n200000_d129_f32"]
    X, y, w_true = workloads.make_logistic(wl.N, wl.D, w_scale=wl.w_scale, key=wl.data_seed,
                                           dtype=wl.dtype)
    rng = np.random.default_rng(11)
    W = w_true[None, :] + rng.normal(0.0, 0.01, size=(wl.num_chains, wl.D))
    say("batched potential full size", wl.N, wl.D, wl.num_chains)
    d = sampler.data(X, y)
    U, G = d.potential_grad(W, batched=True)
    pick = [0, 1, 127, 128, 255]
    _check_potential(orc, X, y, W[pick], U[pick], G[pick])
    # and the streaming kernel agrees on every position
    U2, G2 = d.potential_grad(W)
    np.testing.assert_allclose(U, U2, rtol=1e-6)


def test_batched_potential_rejects(sampler):
    import paper_1912_11554_amd as nuts
    X, y, _ = _data(100, 133, [71, 1])
    say("batched potential rejects")
    d = sampler.data(X, y)
    with pytest.raises(nuts.NutsError) as e:
        d.potential_grad(np.zeros((3, 133)), batched=True)
    assert e.value.code == nuts.NUTS_EUNSUPPORTED
    X64, y64, _ = workloads.make_logistic(100, 10, w_scale=0.3, key=[71, 2])
    d64 = sampler.data(X64, y64)
    with pytest.raises(nuts.NutsError) as e:
        d64.potential_grad(np.zeros((3, 10)), batched=True)
    assert e.value.code == nuts.NUTS_EUNSUPPORTED


def _compare_decisions(gpu, ref, c, atol):
    st, rst = gpu["stats"][c], ref["stats"]
    for f in DECISION_FIELDS:
        bad = np.flatnonzero(st[f] != rst[f])
        assert bad.size == 0, f"chain {c}: {f} differs first at iteration {bad[0]}"
    np.testing.assert_allclose(gpu["samples"][c], ref["samples"], rtol=atol, atol=atol)
    np.testing.assert_allclose(st["potential_energy"], rst["potential_energy"], rtol=1e-6)


@pytest.mark.parametrize("N,D,C,iters,check", [
    (500, 129, 24, 6, range(24)),
    (100, 20, 130, 3, [0, 1, 64, 127, 128, 129]),     # two tiles, the second nearly empty
    (60, 9, 300, 3, [0, 255, 256, 299]),              # two launches (256 + 44 chains)
    (20000, 33, 16, 3, [0, 7, 15]),                   # many stages per group
])
def test_batch_sampler_matches_oracle(sampler, orc, N, D, C, iters, check):
    X, y, _ = _data(N, D, [72, N * 1000 + D])
    step = 0.02 if N <= 1000 else 0.004
    say("batch sampler", N, D, C, iters)
    d = sampler.data(X, y)
    r = d.sample(step_size=step, max_tree_depth=6, num_warmup=1, num_samples=iters - 1,
                 num_chains=C, seed=9, path=3)
    tot = 0
    for c in check:
        ref = orc.nuts(X.astype(np.float64), y, step_size=step, max_tree_depth=6, num_warmup=1,
                       num_samples=iters - 1, seed=9, chain=c)
        _compare_decisions(r, ref, c, atol=1e-5)
        tot += ref["grad_evals"]
    assert r["grad_evals"] > 0


def test_batch_sampler_full_size_ten_iterations(sampler, orc):
    # the 256-chain workload at full size in the benchmark's launch shape (two
    # tiles of 128 chains), every chain started at the generating weights;
    # ten iterations of eight chains spread over both tiles checked one by one
    import concurrent.futures
    import os

    wl = workloads.WORKLOADS["shared256_n200000_d129_f32"]
    X, y, w_true = workloads.make_logistic(wl.N, wl.D, w_scale=wl.w_scale, key=wl.data_seed,
                                           dtype=wl.dtype)
    C, iters = wl.num_chains, 10
    q0 = np.tile(w_true, (C, 1))
    say("batch sampler full size", wl.N, wl.D, C, "iters", iters)
    d = sampler.data(X, y)
    r = d.sample(step_size=wl.step_size, max_tree_depth=wl.max_tree_depth, num_warmup=0,
                 num_samples=iters, num_chains=C, seed=wl.seed, init_q=q0, path=3)
    # every chain: evaluations = 1 + steps of its iterations
    assert r["grad_evals"] == C + int(r["stats"]["num_steps"].sum())
    d.free()
    picks = [0, 37, 64, 127, 128, 150, 201, 255]
    X64 = X.astype(np.float64)
    del X

    def ref(c):
        return orc.nuts(X64, y, step_size=wl.step_size, max_tree_depth=wl.max_tree_depth,
                        num_warmup=0, num_samples=iters, seed=wl.seed, chain=c, init_q=w_true)

    workers = max(1, min(len(picks), len(os.sched_getaffinity(0))))
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        refs = list(ex.map(ref, picks))
    for c, rf in zip(picks, refs):
        _compare_decisions(r, rf, c, atol=1e-5)


def test_batch_sampler_auto_and_resume(sampler):
    # AUTO picks the batch path for many chains on large fp32 data; a run
    # split in two calls (final state, first_iter) equals one call
    X, y, _ = _data(5000, 60, [73, 1])
    say("batch sampler auto/resume")
    d = sampler.data(X, y)
    kw = dict(step_size=0.01, max_tree_depth=5, num_chains=20, seed=5)
    full = d.sample(num_warmup=0, num_samples=6, **kw)
    forced = d.sample(num_warmup=0, num_samples=6, path=3, **kw)
    np.testing.assert_array_equal(full["samples"], forced["samples"])
    a = d.sample(num_warmup=0, num_samples=3, path=3, **kw)
    b = d.sample(num_warmup=0, num_samples=3, path=3, init_q=a["final_q"], first_iter=3, **kw)
    np.testing.assert_array_equal(np.concatenate([a["samples"], b["samples"]], axis=1),
                                  full["samples"])
