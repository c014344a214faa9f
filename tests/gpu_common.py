"""Shared helpers of the GPU parity tests (imported by tests only)."""
import sys

import numpy as np


def say(*a):
    """Name the case before a GPU step so that a crash log says what ran."""
    print("[gpu-case]", *a, file=sys.stderr, flush=True)


def grad_tol(X, w, g_ref, prior_scale, rtol):
    """Per-component bound for a sum of N terms: rtol times the magnitude of
    the summands (|x_ij| with |residual| <= 1, the prior term) plus |g|."""
    X64 = np.asarray(X, dtype=np.float64)
    return rtol * (np.abs(g_ref) + np.abs(X64).sum(axis=0) + np.abs(w) / prior_scale**2 + 1.0)


DECISION_FIELDS = ("tree_depth", "num_steps", "proposal_index", "term_leaf", "direction_bits",
                   "diverging", "turning", "hit_max_depth")


def compare_chain(gpu_samples, gpu_stats, ref, atol=1e-9, accept_atol=None):
    """Decisions bit-exact, positions and energies within atol (relative to
    magnitude), the mean acceptance statistic within accept_atol (default
    atol).  Returns the number of iterations compared."""
    rs, rst = ref["samples"], ref["stats"]
    n = len(rst)
    for f in DECISION_FIELDS:
        bad = np.flatnonzero(gpu_stats[f][:n] != rst[f])
        assert bad.size == 0, f"{f} differs first at iteration {bad[0]}: gpu {gpu_stats[f][bad[0]]} ref {rst[f][bad[0]]}"
    np.testing.assert_allclose(gpu_samples[:n], rs, rtol=atol, atol=atol)
    for f in ("potential_energy", "energy"):
        np.testing.assert_allclose(gpu_stats[f][:n], rst[f], rtol=atol, atol=atol)
    ta = atol if accept_atol is None else accept_atol
    np.testing.assert_allclose(gpu_stats["accept_prob"][:n], rst["accept_prob"], rtol=ta, atol=ta)
    return n
