"""Pins for the iterative tree builder's index logic (Appendix A, Alg. 2).

The candidate set C(n) is checked against a brute-force enumeration of the
balanced subtrees that end at leaf n, against the paper's worked example for
n = 11, and against the S-array invariant; the checks the oracle actually
performs are read back from its trace.
"""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_force_candidates(n):
    """First leaves of every aligned block [a, n] of size 2^m >= 2 that ends
    at leaf n, smallest block first."""
    out = []
    m = 1
    while (1 << m) <= n + 1:
        size = 1 << m
        if (n + 1) % size == 0:
            out.append(n - size + 1)
        m += 1
    return out


def test_bitcount_trailing_ones(orc):
    for n in range(4096):
        assert orc.bitcount(n) == bin(n).count("1")
        assert orc.trailing_ones(n) == len(bin(n)) - len(bin(n).rstrip("1"))


def test_worked_example_n11(orc):
    g = json.load(open(os.path.join(GOLDEN, "uturn_candidates_n11.json")))
    n = g["n"]
    i_max, i_min = orc.check_range(n)
    assert orc.trailing_ones(n) == g["trailing_ones"]
    assert i_max - i_min + 1 == len(g["candidates"])
    # slot i holds the largest even k < n with BitCount(k) = i
    slots = {}
    for k in range(0, n, 2):
        slots[orc.bitcount(k)] = k
    assert [slots[i] for i in range(i_max, i_min - 1, -1)] == g["candidates"]
    assert brute_force_candidates(n) == g["candidates"]


@pytest.mark.parametrize("d", range(1, 11))
def test_candidate_slots_all_n(orc, d):
    for n in range(1, 1 << d, 2):
        i_max, i_min = orc.check_range(n)
        slots = {}
        for k in range(0, n, 2):
            slots[orc.bitcount(k)] = k
        got = [slots[i] for i in range(i_max, i_min - 1, -1)]
        assert got == brute_force_candidates(n)
        # the S array never needs more than d slots
        assert i_max <= d - 1


def _straight_line_run(orc, builder, depth):
    # Prior-only target (X = 0 logistic) with a tiny step: trajectories are
    # nearly straight, no subtree ever U-turns, every check is performed.
    D = 2
    X = np.zeros((1, D))
    y = np.zeros(1, dtype=np.uint8)
    return orc.nuts(X, y, step_size=1e-7, max_tree_depth=depth, num_warmup=0, num_samples=1,
                    seed=5, builder=builder, init_q=np.array([3.0, -2.0]), trace_cap=1 << 14)


@pytest.mark.parametrize("builder", [0, 1])
def test_trace_matches_brute_force(orc, builder):
    depth = 10
    r = _straight_line_run(orc, builder, depth)
    st = r["stats"][0]
    assert st["hit_max_depth"] == 1 and st["tree_depth"] == depth
    assert st["num_steps"] == (1 << depth) - 1
    tr = r["trace"]
    # expected: for every doubling j, for every odd leaf n < 2^j, the
    # candidates of n in order, as pairs (first leaf, n)
    want = []
    for j in range(depth):
        for n in range(1, 1 << j, 2):
            want += [(a, n) for a in brute_force_candidates(n)]
    assert [tuple(x) for x in tr] == want
