"""Effective sample size and Monte Carlo standard error -- TEST INFRASTRUCTURE.

The paper reports ESS without defining it.  This module uses Geyer's
initial monotone sequence estimator (Geyer, "Practical Markov chain Monte
Carlo", Stat. Sci. 1992) on autocorrelations from an FFT, and for several
chains the multi-chain form of Gelman et al., BDA3 section 11.5 (within- and
between-chain variances).  Plain numpy.
"""
from __future__ import annotations

import numpy as np


def autocovariance(x):
    """Biased autocovariance at all lags of a 1-D series, via zero-padded FFT."""
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[0]
    xc = x - x.mean()
    m = 1
    while m < 2 * n:
        m *= 2
    f = np.fft.rfft(xc, n=m)
    acov = np.fft.irfft(f * np.conj(f), n=m)[:n]
    return acov / n


def ess(chains):
    """ESS of one scalar quantity.  ``chains`` is [n] or [C, n]."""
    x = np.asarray(chains, dtype=np.float64)
    if x.ndim == 1:
        x = x[None, :]
    C, n = x.shape
    if n < 4:
        return float(C * n)
    acov = np.stack([autocovariance(x[c]) for c in range(C)])
    chain_mean = x.mean(axis=1)
    w = acov[:, 0].mean() * n / (n - 1.0)          # within-chain variance
    var_plus = w * (n - 1.0) / n
    if C > 1:
        var_plus += chain_mean.var(ddof=1)          # between-chain term B/n
    if not var_plus > 0:
        return float(C * n)
    rho = 1.0 - (w - acov.mean(axis=0)) / var_plus  # combined autocorrelation
    rho[0] = 1.0
    # Geyer: sums of adjacent pairs are positive and non-increasing
    tau = -1.0
    prev = np.inf
    t = 0
    while t + 1 < n:
        pair = rho[t] + rho[t + 1]
        if pair <= 0:
            break
        pair = min(pair, prev)
        prev = pair
        tau += 2.0 * pair
        t += 2
    # Strongly antithetic chains can drive the Geyer sum below zero; bound
    # tau from below as Stan and ArviZ do (Vehtari et al. 2021).
    tau = max(tau, 1.0 / np.log10(C * n))
    return float(C * n / tau)


def ess_columns(samples):
    """Per-coordinate ESS of samples [n, D] or [C, n, D]."""
    s = np.asarray(samples, dtype=np.float64)
    if s.ndim == 2:
        s = s[None]
    return np.array([ess(s[:, :, d]) for d in range(s.shape[2])])


def mcse_mean(samples):
    """Monte Carlo standard error of the mean of each coordinate."""
    s = np.asarray(samples, dtype=np.float64)
    flat = s.reshape(-1, s.shape[-1])
    return flat.std(axis=0, ddof=1) / np.sqrt(ess_columns(s))
