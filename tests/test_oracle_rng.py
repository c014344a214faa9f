"""Pins for the oracle's counter-based RNG.

Philox4x64-10 is pinned to numpy's independent implementation
(``numpy.random.Philox``, which produces the block of counter c+1 when its
state holds counter c).  The uniform and normal transforms are pinned by
range, by inverting Box-Muller, and by distribution tests.
"""
import numpy as np
import pytest
from scipy import stats


def _numpy_block(counter, key):
    c = np.array(counter, dtype=object)
    # numpy increments its 256-bit counter before producing a block
    val = int(c[0]) | (int(c[1]) << 64) | (int(c[2]) << 128) | (int(c[3]) << 192)
    val = (val - 1) % (1 << 256)
    words = [(val >> (64 * i)) & ((1 << 64) - 1) for i in range(4)]
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array(words, dtype=np.uint64))
    return bg.random_raw(4)


@pytest.mark.parametrize("counter,key", [
    ([1, 0, 0, 0], [0, 0]),
    ([0, 0, 0, 0], [5, 7]),
    ([7, (1 << 32) | 3, 12, 0], [0, 0]),
    ([123456789, (4 << 32) | 9, 1023, 0], [42, 4095]),
    ([2**64 - 1, 2**64 - 1, 2**64 - 1, 2**64 - 1], [2**64 - 1, 2**63]),
    ([0, 0, 0, 1], [1, 2]),
])
def test_philox_matches_numpy(orc, counter, key):
    got = orc.philox4x64_10(counter, key)
    want = _numpy_block(counter, key)
    assert np.array_equal(got, want)


def test_philox_many_random_counters(orc):
    rng = np.random.default_rng(11)
    for _ in range(200):
        counter = [int(x) for x in rng.integers(0, 2**63, size=4, dtype=np.int64)]
        key = [int(x) for x in rng.integers(0, 2**63, size=2, dtype=np.int64)]
        assert np.array_equal(orc.philox4x64_10(counter, key), _numpy_block(counter, key))


def test_u53_range_and_resolution(orc):
    assert orc.u53(0) == 0.0
    assert orc.u53(2**64 - 1) == 1.0 - 2.0**-53
    assert orc.u53(1 << 11) == 2.0**-53
    assert orc.u53((1 << 11) - 1) == 0.0


def test_normals_invert_box_muller(orc):
    # each pair (n0, n1) satisfies n0^2 + n1^2 = -2 ln(1 - ua) and has polar
    # angle 2 pi ub, with (ua, ub) the uniforms of the Philox block
    seed, chain, t, D = 3, 17, 41, 13
    z = orc.normals(seed, chain, t, D)
    for b in range(4):
        w = orc.philox4x64_10([t, (1 << 32) | 0, b, 0], [seed, chain])
        u = [orc.u53(int(x)) for x in w]
        for pair in range(2):
            i0 = 4 * b + 2 * pair
            if i0 + 1 >= D:
                continue
            r2 = z[i0] ** 2 + z[i0 + 1] ** 2
            assert r2 == pytest.approx(-2.0 * np.log1p(-u[2 * pair]), rel=1e-13)
            ang = np.arctan2(z[i0 + 1], z[i0]) % (2 * np.pi)
            assert ang == pytest.approx(2 * np.pi * u[2 * pair + 1], abs=1e-12)


def test_normals_distribution(orc):
    D = 16
    draws = np.concatenate([orc.normals(1, 2, t, D) for t in range(4000)])
    assert abs(draws.mean()) < 4.0 / np.sqrt(draws.size)
    assert draws.var() == pytest.approx(1.0, abs=5 * np.sqrt(2.0 / draws.size))
    assert stats.kstest(draws, "norm").pvalue > 1e-3


def test_normals_prefix_stable(orc):
    # momentum coordinate i does not depend on the dimension D it is drawn for
    a = orc.normals(9, 1, 5, 7)
    b = orc.normals(9, 1, 5, 257)
    assert np.array_equal(a, b[:7])


def test_direction_and_uniform_draws(orc):
    dirs = np.array([orc.direction(0, c, t, j) for c in range(4) for t in range(100)
                     for j in range(10)])
    assert set(np.unique(dirs)) == {-1, 1}
    assert abs((dirs > 0).mean() - 0.5) < 4 * 0.5 / np.sqrt(dirs.size)
    um = np.array([orc.u_merge(0, 0, t, j) for t in range(300) for j in range(10)])
    ul = np.array([orc.u_leaf(0, 0, 7, 9, n) for n in range(3000)])
    for u in (um, ul):
        assert u.min() >= 0.0 and u.max() < 1.0
        assert stats.kstest(u, "uniform").pvalue > 1e-3
    # the tags keep the streams apart
    assert orc.u_merge(0, 0, 5, 3) != orc.u_leaf(0, 0, 5, 3, 0)


def test_tree_draws_come_from_the_documented_words(orc):
    # reading R8: block b of tag 2 (counter {t, 2 << 32, b, 0}, key {seed,
    # chain}) holds the direction of doubling b (word 0, low bit), the merge
    # uniform of doubling b (word 1) and the uniforms of leaves 2b, 2b + 1
    # (words 2, 3), leaf n of doubling j being number 2^j - 1 + n; the words
    # are taken from numpy's Philox, not from the oracle's
    seed, chain, t = 9, 33, 1234
    u53 = lambda w: float(int(w) >> 11) * 2.0**-53
    for j in range(12):
        w = _numpy_block([t, 2 << 32, j, 0], [seed, chain])
        assert orc.direction(seed, chain, t, j) == (1 if int(w[0]) & 1 else -1)
        assert orc.u_merge(seed, chain, t, j) == u53(w[1])
    for j, n in [(0, 0), (1, 0), (1, 1), (2, 3), (6, 0), (7, 0), (7, 127), (9, 300), (20, 12345)]:
        g = (1 << j) - 1 + n
        w = _numpy_block([t, 2 << 32, g >> 1, 0], [seed, chain])
        assert orc.u_leaf(seed, chain, t, j, n) == u53(w[2 + (g & 1)])
