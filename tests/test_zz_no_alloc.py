"""The allocation-free potential entry point (nuts_data_potential_grad_noalloc)
against the allocating one it mirrors (nuts_data_potential_grad), through
the C ABI: the same kernel on the same plan, so the results must be bitwise
identical.  Two calls in a row, the second on a smaller input, then the
first input again, and the rejections (host memory, a request larger than
the fixed workspace)."""
import numpy as np
import pytest

import workloads
from tests.gpu_common import say

pytestmark = pytest.mark.gpu


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _both(d, W, s=1.0):
    import torch
    K = W.shape[0]
    Wd = _dev(W)
    U0 = torch.zeros(K, dtype=torch.float64, device="cuda")
    G0 = torch.zeros((K, d.D), dtype=torch.float64, device="cuda")
    U1 = torch.full((K,), np.nan, dtype=torch.float64, device="cuda")
    G1 = torch.full((K, d.D), np.nan, dtype=torch.float64, device="cuda")
    d.potential_grad(Wd, prior_scale=s, out_U=U0, out_grad=G0)
    d.potential_grad(Wd, prior_scale=s, out_U=U1, out_grad=G1, no_alloc=True)
    torch.cuda.synchronize()
    return U0.cpu().numpy(), G0.cpu().numpy(), U1.cpu().numpy(), G1.cpu().numpy()


def test_noalloc_matches_allocating_entry_point():
    import torch

    import paper_1912_11554_amd as nuts
    s = nuts.Sampler(0)
    # call 1: a larger fp32 data set (ragged last block), three positions
    X1, y1, w1 = workloads.make_logistic(100_003, 55, w_scale=0.5, key=[95, 1], dtype="f32")
    d1 = s.data(_dev(X1), _dev(y1))
    W1 = w1[None, :] + np.random.default_rng(1).normal(0.0, 0.05, size=(3, 55))
    say("noalloc call 1", X1.shape, "K", 3)
    U0, G0, U1, G1 = _both(d1, W1)
    assert np.array_equal(U0, U1) and np.array_equal(G0, G1)
    # call 2: a smaller fp64 data set, one position, another prior scale
    X2, y2, w2 = workloads.make_logistic(3001, 9, w_scale=1.0, key=[95, 2])
    d2 = s.data(_dev(X2), _dev(y2))
    say("noalloc call 2", X2.shape, "K", 1)
    U0, G0, U1, G1 = _both(d2, w2[None, :], s=2.0)
    assert np.array_equal(U0, U1) and np.array_equal(G0, G1)
    # and back to the first data set with more positions than CUs' groups
    W3 = w1[None, :] + np.random.default_rng(3).normal(0.0, 0.05, size=(300, 55))
    say("noalloc call 3", X1.shape, "K", 300)
    U0, G0, U1, G1 = _both(d1, W3)
    assert np.array_equal(U0, U1) and np.array_equal(G0, G1)
    # per-chain data sets: one position per data set
    wl = workloads.WORKLOADS["chains4096_n500_d9_f64"]
    Xc, yc = workloads.make_workload(wl, chains=range(64))
    dc = s.data(_dev(Xc), _dev(yc), per_chain=True)
    say("noalloc per-chain K", 64)
    U0, G0, U1, G1 = _both(dc, np.random.default_rng(4).normal(size=(64, 9)))
    assert np.array_equal(U0, U1) and np.array_equal(G0, G1)

    # rejections: host memory, and more partial sums than the workspace holds
    with pytest.raises(nuts.NutsError) as e:
        d2.potential_grad(w2[None, :], no_alloc=True)
    assert e.value.code == nuts.NUTS_EINVAL
    Wbig = torch.zeros((9000, 55), dtype=torch.float64, device="cuda")
    Ub = torch.zeros(9000, dtype=torch.float64, device="cuda")
    Gb = torch.zeros((9000, 55), dtype=torch.float64, device="cuda")
    with pytest.raises(nuts.NutsError) as e:
        d1.potential_grad(Wbig, out_U=Ub, out_grad=Gb, no_alloc=True)
    assert e.value.code == nuts.NUTS_EINVAL
    assert "fixed workspace" in str(e.value)
    torch.cuda.synchronize()
    for d in (d1, d2, dc):
        d.free()
    s.close()
