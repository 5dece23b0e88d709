"""Pins of the oracle's centered-rank fitness shaping (Sec. 3.2; App. B).

Ranks are checked against numpy's stable argsort (a library routine) on every
tie pattern for small N; the weights against their exact properties.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from oracle import brute
from oracle import oracle as O


def _stable_rank(keys):
    order = np.argsort(keys, kind="stable")
    r = np.empty(len(keys), np.int32)
    r[order] = np.arange(len(keys))
    return r


@pytest.mark.parametrize("N", [2, 3, 4, 5, 6, 7, 8])
def test_ranks_exhaustive_ties(N):
    # every fitness vector over {0,1,2}^N: all tie patterns
    vals = np.array(list(itertools.product([0.0, 1.0, 2.0], repeat=N)), np.float32)
    for f in vals:
        np.testing.assert_array_equal(O.ranks(f), _stable_rank(f))
        np.testing.assert_array_equal(O.ranks(f, maximize=1), _stable_rank(-f))


@pytest.mark.parametrize("N", [2, 4, 6, 7])
def test_ranks_all_permutations(N):
    for perm in itertools.permutations(range(N)):
        f = np.array(perm, np.float32) * np.float32(0.5) - 1
        np.testing.assert_array_equal(O.ranks(f), np.array(perm, np.int32))


def test_ranks_special_values():
    f = np.array([np.nan, -0.0, 0.0, np.inf, -np.inf, 1.0, np.nan, -1.0], np.float32)
    # NaN takes the key +inf (ties with +inf, broken by index); -0 == +0 (tie by index)
    want = [5, 2, 3, 6, 0, 4, 7, 1]
    np.testing.assert_array_equal(O.ranks(f), want)
    assert list(O.ranks(f)) == brute.ranks(list(f))
    # maximising: NaN still worst; -inf (key +inf) now ties with it
    assert list(O.ranks(f, 1)) == brute.ranks(list(f), True)
    np.testing.assert_array_equal(O.ranks(f, 1), [5, 2, 3, 0, 6, 1, 7, 4])


def test_ranks_invariant_under_increasing_transform():
    rng = np.random.default_rng(0)
    f = rng.normal(size=257).astype(np.float32)
    f[10] = f[20]  # a tie
    for g in (3 * f + 7, np.exp(f / 4), f ** 3):
        np.testing.assert_array_equal(O.ranks(g.astype(np.float32)), O.ranks(f))


@pytest.mark.parametrize("N", [2, 4, 8, 32, 64, 256, 1000, 1024, 2048, 4096])
def test_centered_weights_exact_properties(N):
    f = np.arange(N, dtype=np.float32)[::-1].copy()  # distinct; rank_j = N-1-j
    y = O.shape(f)
    y64 = y.astype(np.float64)
    # sum is exactly zero (antisymmetry y(r) = -y(N-1-r) holds bit for bit)
    assert np.sum(y64) == 0.0
    yr = y[::-1]
    np.testing.assert_array_equal(y, -yr)
    assert y.min() == np.float32(-0.5) and y.max() == np.float32(0.5)
    assert np.all(np.abs(y) <= 0.5)
    # each weight is the correctly rounded fp32 of (2r-(N-1))/(2(N-1))
    ranks = O.ranks(f)
    for j in range(0, N, max(1, N // 64)):
        assert y[j] == brute.f32(Fraction(2 * int(ranks[j]) - (N - 1), 2 * (N - 1)))


def test_centered_weights_monotone_in_fitness():
    rng = np.random.default_rng(1)
    f = rng.normal(size=100).astype(np.float32)
    y = O.shape(f)
    order = np.argsort(f, kind="stable")
    assert np.all(np.diff(y[order]) > 0)
    ym = O.shape(f, maximize=1)
    np.testing.assert_array_equal(ym, -y)  # distinct values: maximising mirrors


def test_raw_shaping_is_key():
    f = np.array([3.0, -1.0, 2.5, 0.0], np.float32)
    np.testing.assert_array_equal(O.shape(f, 0, O.SHAPE_RAW), f)
    np.testing.assert_array_equal(O.shape(f, 1, O.SHAPE_RAW), -f)
