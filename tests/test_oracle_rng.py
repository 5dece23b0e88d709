"""Pins of the oracle's random stream (CPU only).

Philox-4x32-10 against the published known-answer vectors; the uniform and
Box-Muller maps against exactness, the brute-force reference and the normal
distribution (the Gaussian search distribution of Sec. 2.1).
"""
import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle import brute
from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kats():
    rows = []
    with open(GOLDEN) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(w, 16) for w in line.split()]
            rows.append((tuple(v[0:4]), tuple(v[4:6]), tuple(v[6:10])))
    assert len(rows) == 3
    return rows


@pytest.mark.parametrize("ctr,key,want", _kats())
def test_philox_kat_oracle(ctr, key, want):
    assert tuple(O.philox(key, ctr)) == want


@pytest.mark.parametrize("ctr,key,want", _kats())
def test_philox_kat_brute(ctr, key, want):
    assert tuple(brute.philox(key, ctr)) == want


def test_counter_layout_words():
    # words(seed, domain, row, t, b) = Philox(key=(lo,hi of seed), ctr=(b,row,t,domain))
    seed = (7 << 32) | 123
    w = O.words(seed, 2, 5, 9, 3, 2)
    assert list(w[:4]) == brute.philox((123, 7), (3, 5, 9, 2))
    assert list(w[4:]) == brute.philox((123, 7), (4, 5, 9, 2))


def test_normals_match_brute_bits():
    # Two independent Box-Muller implementations agree bit for bit.
    for seed, dom, row, t in [(0, 0, 0, 0), (3, 0, 17, 5), (1023, 1, 0, 0), (2, 2, 0, 0), (5, 3, 0, 11)]:
        got = O.normals(seed, dom, row, t, 0, 24)
        ref = []
        for b in range(6):
            ref += brute.normals_block(seed, dom, row, t, b)
        np.testing.assert_array_equal(got, np.array(ref, np.float32))


def test_normals_offset_window():
    full = O.normals(11, 0, 3, 2, 0, 40)
    for d0, nd in [(1, 5), (3, 9), (4, 4), (37, 3)]:
        np.testing.assert_array_equal(O.normals(11, 0, 3, 2, d0, nd), full[d0:d0 + nd])


def test_uniform_extremes_are_finite():
    # u_pos in (0, 1]: the largest |normal| is sqrt(2*24*ln 2) ~ 5.77, never inf.
    z = O.normals(0, 0, 0, 0, 0, 1 << 18)
    assert np.all(np.isfinite(z))
    assert np.max(np.abs(z)) <= math.sqrt(2 * 24 * math.log(2)) + 1e-6


def test_normal_distribution_moments_and_ks():
    n = 1 << 21
    z = O.normals(42, 0, 0, 0, 0, n).astype(np.float64)
    se = 1.0 / math.sqrt(n)
    assert abs(z.mean()) < 5 * se
    assert abs(z.var() - 1.0) < 5 * math.sqrt(2.0) * se
    assert abs(stats.kurtosis(z, fisher=False) - 3.0) < 5 * math.sqrt(24.0) * se
    assert abs(stats.skew(z)) < 5 * math.sqrt(6.0) * se
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # consecutive draws (both Box-Muller partners and different blocks) uncorrelated
    for lag in (1, 2, 3, 4):
        c = np.corrcoef(z[:-lag], z[lag:])[0, 1]
        assert abs(c) < 5 * se


def test_streams_are_distinct():
    # different rows (pairs), generations, domains and seeds give unrelated draws
    base = O.normals(0, 0, 0, 0, 0, 4096).astype(np.float64)
    for args in [(0, 0, 1, 0), (0, 0, 0, 1), (0, 1, 0, 0), (1, 0, 0, 0)]:
        other = O.normals(*args, 0, 4096).astype(np.float64)
        assert abs(np.corrcoef(base, other)[0, 1]) < 5 / 64.0


def test_antithetic_pairs_sum_to_zero():
    # Perturbation rows j and j+N/2 are exact negatives (antithetic sampling,
    # Sec. 2.1): with m = 0 the members themselves are exact negatives.
    cfg = O.OracleConfig(num_dims=10, popsize=8, init=O.INIT_ZERO, sigma=0.37, seed=4)
    x = O.population(cfg, 0, 3, np.zeros(10, np.float32))
    np.testing.assert_array_equal(x[:4] + x[4:], np.zeros((4, 10), np.float32))
    eps = np.stack([O.noise(cfg, 0, 3, p) for p in range(4)])
    np.testing.assert_array_equal(x[:4], np.float32(0.37) * eps)


def test_init_uniform_matches_brute_and_range():
    cfg = O.OracleConfig(num_dims=13, popsize=2, init=O.INIT_UNIFORM, init_lo=-5.12, init_hi=5.12, seed=9)
    m = O.init_mean(cfg, 0)
    ref = brute.init_uniform(9, 13, -5.12, 5.12)
    np.testing.assert_array_equal(m, np.array(ref, np.float32))
    big = O.OracleConfig(num_dims=1 << 16, popsize=2, init=O.INIT_UNIFORM, init_lo=-2, init_hi=2, seed=1)
    mb = O.init_mean(big, 0)
    assert mb.min() >= -2 and mb.max() < 2
    assert abs(mb.mean()) < 5 * (4 / math.sqrt(12)) / 256


def test_batch_run_r_uses_seed_plus_r():
    # A run r of an R-batch equals a standalone run whose seed is seed + r
    # (independent keys per run, Listing 3's vmap over keys).
    cfg = O.OracleConfig(num_dims=6, popsize=4, num_runs=3, seed=10, problem=O.PROB_SPHERE)
    es = O.OracleES(cfg)
    es.run(3)
    for r in range(3):
        solo = O.OracleES(O.OracleConfig(num_dims=6, popsize=4, num_runs=1, seed=10 + r, problem=O.PROB_SPHERE))
        solo.run(3)
        np.testing.assert_array_equal(es.m[r], solo.m[0])
