"""Sample diagnostics for the benchmark: effective sample size per coordinate.

Geyer's initial monotone sequence estimator (Stat. Sci. 1992): the
autocorrelations of each coordinate are summed in adjacent pairs while the
pair sums stay positive, each pair capped by the previous one; several chains
are combined through the within/between-chain variance of Gelman et al.
(BDA3, section 11.5).  Works on all coordinates at once.
"""
from __future__ import annotations

import numpy as np


def effective_sample_size(draws) -> np.ndarray:
    """draws: [n, D] (one chain) or [C, n, D].  Returns ESS per coordinate."""
    x = np.asarray(draws, dtype=np.float64)
    if x.ndim == 2:
        x = x[None]
    C, n, D = x.shape
    if n < 4:
        return np.full(D, float(C * n))
    centred = x - x.mean(axis=1, keepdims=True)
    size = 1 << int(np.ceil(np.log2(2 * n)))
    spec = np.fft.rfft(centred, n=size, axis=1)
    acov = np.fft.irfft(spec * spec.conj(), n=size, axis=1)[:, :n, :] / n   # [C, n, D]
    within = acov[:, 0, :].mean(axis=0) * n / (n - 1.0)
    var_hat = within * (n - 1.0) / n
    if C > 1:
        var_hat = var_hat + x.mean(axis=1).var(axis=0, ddof=1)
    safe = np.where(var_hat > 0, var_hat, 1.0)
    rho = 1.0 - (within[None, :] - acov.mean(axis=0)) / safe[None, :]     # [n, D]
    rho[0] = 1.0
    npairs = n // 2
    pairs = rho[: 2 * npairs].reshape(npairs, 2, D).sum(axis=1)           # [npairs, D]
    positive = np.cumprod(pairs > 0, axis=0).astype(bool)                 # initial positive run
    capped = np.minimum.accumulate(np.where(positive, pairs, np.inf), axis=0)
    tau = -1.0 + 2.0 * np.where(positive, capped, 0.0).sum(axis=0)
    tau = np.maximum(tau, 1.0 / np.log10(C * n))
    ess = C * n / tau
    return np.where(var_hat > 0, ess, float(C * n))


def effective_sample_size_per_chain(draws) -> np.ndarray:
    """draws: [C, n, D] from C chains with different targets.  Returns the
    single-chain ESS of every (chain, coordinate), shape [C, D]."""
    x = np.asarray(draws, dtype=np.float64)
    C, n, D = x.shape
    flat = np.transpose(x, (1, 0, 2)).reshape(n, C * D)
    return effective_sample_size(flat).reshape(C, D)
