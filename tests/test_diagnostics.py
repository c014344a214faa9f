"""The package's ESS (used by the benchmark) agrees with the oracle's ESS
and with the AR(1) closed form."""
import numpy as np
import pytest

from oracle.ess import ess
from paper_1912_11554_amd.diagnostics import effective_sample_size


def _ar1(phi, n, rng, C=1, D=3):
    e = rng.normal(size=(C, n, D))
    x = np.zeros((C, n, D))
    x[:, 0] = e[:, 0]
    for t in range(1, n):
        x[:, t] = phi * x[:, t - 1] + np.sqrt(1 - phi * phi) * e[:, t]
    return x


@pytest.mark.parametrize("phi,C", [(0.0, 1), (0.7, 1), (0.9, 4), (-0.5, 2)])
def test_matches_oracle_and_closed_form(phi, C):
    rng = np.random.default_rng(int(10 * abs(phi)) + C)
    x = _ar1(phi, 20000, rng, C=C)
    got = effective_sample_size(x if C > 1 else x[0])
    for d in range(3):
        assert got[d] == pytest.approx(ess(x[:, :, d]), rel=1e-9)
    want = C * 20000 * (1 - phi) / (1 + phi)
    assert np.all(np.abs(got / want - 1) < 0.2)


def test_per_chain_ess_matches_single_chain_calls():
    from paper_1912_11554_amd.diagnostics import effective_sample_size_per_chain
    rng = np.random.default_rng(9)
    x = np.stack([_ar1(phi, 4000, rng, D=1)[0, :, 0] for phi in (0.1, 0.5, 0.8)])   # [3, n]
    draws = np.stack([x, -x], axis=2)                                       # [3, n, 2]
    got = effective_sample_size_per_chain(draws)
    for c in range(3):
        assert got[c, 0] == pytest.approx(effective_sample_size(draws[c])[0], rel=1e-12)
    assert got[0, 0] > got[2, 0]
