"""Seeded synthetic workloads shaped like the paper's logistic-regression runs.

This module only draws inputs; it holds none of the sampler's arithmetic.
Both the CPU oracle side (tests, CPU baseline) and the GPU side (tests,
bench) take their inputs from here, so the two always see identical arrays.

Recipe (one numpy ``Generator(Philox(key=data_seed))`` per dataset):
  1. w_true ~ N(0, w_scale^2) over all D columns (the intercept included);
  2. X: N x (D-1) iid N(0, 1) features, optionally zeroed at random with
     probability ``zero_frac``, then a final column of ones (the intercept);
  3. y_i ~ Bernoulli(sigmoid(x_i . w_true)).
Rows are drawn in fixed-size chunks, so large datasets never need a full
fp64 temporary, and the result does not depend on the output dtype.

Forest CoverType (581,012 x 54 normalised features, binary labels) is not
available here; iid standard-normal features of the same shape stand in for it.
"""
from __future__ import annotations

import dataclasses

import numpy as np

CHUNK_ROWS = 1 << 16


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    N: int
    D: int                 # including the intercept column
    dtype: str             # "f64" or "f32"
    w_scale: float
    data_seed: int
    step_size: float
    max_tree_depth: int
    num_warmup: int
    num_samples: int
    num_chains: int = 1
    per_chain_data: bool = False
    zero_frac: float = 0.0
    adapt_diag_mass: bool = False
    prior_scale: float = 1.0
    seed: int = 0


WORKLOADS = {
    # small single chain (latency-bound correctness case)
    "logreg_n1000_d11_f64": Workload("logreg_n1000_d11_f64", 1000, 11, "f64", 1.0, 1,
                                     0.05, 10, 200, 200),
    # covtype-shaped single chain, fp64 and fp32
    "covtype_n581012_d55_f64": Workload("covtype_n581012_d55_f64", 581012, 55, "f64", 0.5, 2,
                                        0.0015, 10, 1000, 1000),
    "covtype_n581012_d55_f32": Workload("covtype_n581012_d55_f32", 581012, 55, "f32", 0.5, 2,
                                        0.0015, 10, 1000, 1000),
    # 4096 independent small chains, each with its own data
    "chains4096_n500_d9_f64": Workload("chains4096_n500_d9_f64", 500, 9, "f64", 1.0, 3,
                                       0.1, 8, 500, 500, num_chains=4096, per_chain_data=True),
    # 256 chains sharing one dataset
    "shared256_n200000_d129_f32": Workload("shared256_n200000_d129_f32", 200000, 129, "f32",
                                           0.3, 4, 0.002, 10, 500, 500, num_chains=256),
    # large streaming single chain with 10% of feature entries zeroed
    "stream_n4m_d257_f32": Workload("stream_n4m_d257_f32", 4000000, 257, "f32", 0.1, 5,
                                    0.0005, 10, 300, 300, zero_frac=0.1, adapt_diag_mass=True),
}


def _np_dtype(dtype: str):
    return {"f64": np.float64, "f32": np.float32}[dtype]


def make_logistic(N: int, D: int, *, w_scale: float, key, dtype: str = "f64",
                  zero_frac: float = 0.0):
    """Draw (X [N, D] row-major with a trailing ones column, y [N] uint8,
    w_true [D]) from a Philox generator keyed by ``key``."""
    rng = np.random.Generator(np.random.Philox(key=key))
    w_true = rng.normal(0.0, w_scale, size=D)
    X = np.empty((N, D), dtype=_np_dtype(dtype))
    y = np.empty(N, dtype=np.uint8)
    for r0 in range(0, N, CHUNK_ROWS):
        r1 = min(N, r0 + CHUNK_ROWS)
        feats = rng.normal(size=(r1 - r0, D - 1))
        if zero_frac > 0.0:
            feats *= rng.random(size=feats.shape) >= zero_frac
        blk = np.empty((r1 - r0, D), dtype=np.float64)
        blk[:, : D - 1] = feats
        blk[:, D - 1] = 1.0
        X[r0:r1] = blk
        eta = blk @ w_true
        prob = 1.0 / (1.0 + np.exp(-eta))
        y[r0:r1] = rng.random(size=r1 - r0) < prob
    return X, y, w_true


def make_workload(wl: Workload, *, chains=None, rows=None):
    """Inputs for a workload.  Shared data: (X [N, D], y [N]).  Per-chain
    data: (X [C, N, D], y [C, N]) for the chain indices in ``chains``
    (default all), chain c keyed by (data_seed, c).  ``rows`` truncates N."""
    N = wl.N if rows is None else min(rows, wl.N)
    if not wl.per_chain_data:
        X, y, _ = make_logistic(N, wl.D, w_scale=wl.w_scale, key=wl.data_seed, dtype=wl.dtype,
                                zero_frac=wl.zero_frac)
        return X, y
    idx = range(wl.num_chains) if chains is None else chains
    Xs, ys = [], []
    for c in idx:
        X, y, _ = make_logistic(N, wl.D, w_scale=wl.w_scale, key=[wl.data_seed, int(c)],
                                dtype=wl.dtype, zero_frac=wl.zero_frac)
        Xs.append(X)
        ys.append(y)
    return np.stack(Xs), np.stack(ys)


def make_lingauss(N: int, D: int, *, key, noise_scale: float = 1.0):
    """Linear-Gaussian regression data (X [N, D], y [N] float) for the
    conjugate-posterior tests of the sampler."""
    rng = np.random.Generator(np.random.Philox(key=key))
    w_true = rng.normal(size=D)
    X = rng.normal(size=(N, D))
    yv = X @ w_true + noise_scale * rng.normal(size=N)
    return X, yv


def make_hmm(T: int = 600, Tsup: int = 100, K: int = 3, V: int = 10, *, key=6, stay: float = 0.7,
             emit_conc: float = 0.5):
    """A semi-supervised HMM data set shaped like the paper's HMM benchmark
    (K = 3 hidden states, V = 10 symbols, T = 600 points, the first 100 hidden
    states observed).  The paper does not give its fixed matrices; here the
    transition matrix keeps the state with probability ``stay`` and moves to
    each other state equally, and the emission rows are Dirichlet(emit_conc)
    draws.  Returns (w [T] uint8, z [Tsup] uint8, theta [K, K], phi [K, V])."""
    rng = np.random.Generator(np.random.Philox(key=key))
    theta = np.full((K, K), (1.0 - stay) / (K - 1))
    np.fill_diagonal(theta, stay)
    phi = rng.dirichlet(np.full(V, emit_conc), size=K)
    z = np.empty(T, dtype=np.int64)
    z[0] = rng.integers(K)
    for t in range(1, T):
        z[t] = rng.choice(K, p=theta[z[t - 1]])
    w = np.array([rng.choice(V, p=phi[k]) for k in z], dtype=np.uint8)
    return w, z[:Tsup].astype(np.uint8), theta, phi
