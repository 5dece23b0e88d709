"""The oracle against the independent brute-force reference on tiny problems
(D <= 4, N <= 8), stage by stage over 50 generations, for every problem.

At each generation both sides start from the brute-force state, so a single
rounding difference cannot snowball into a different trajectory."""
import math

import numpy as np
import pytest

from oracle import brute
from oracle import oracle as O

PROBS = [("sphere", O.PROB_SPHERE, -5.0, 5.0), ("rosenbrock", O.PROB_ROSENBROCK, -2.0, 2.0),
         ("rastrigin", O.PROB_RASTRIGIN, -5.12, 5.12), ("shifted_sphere", O.PROB_SHIFTED_SPHERE, -1.0, 1.0)]


def _ulps(a, b):
    a, b = np.float32(a), np.float32(b)
    return abs(float(a) - float(b)) / float(np.spacing(np.float32(max(abs(a), abs(b), 1e-30))))


@pytest.mark.parametrize("name,prob,lo,hi", PROBS)
@pytest.mark.parametrize("D", [1, 2, 3, 4])
@pytest.mark.parametrize("N", [2, 4, 6, 8])
def test_oracle_matches_brute(name, prob, lo, hi, D, N):
    seed = 100 * D + N
    sigma, lr = 0.1, 0.05
    cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=sigma, lr=lr, seed=seed, init=O.INIT_UNIFORM,
                         init_lo=lo, init_hi=hi, problem=prob)
    es = O.OracleES(cfg)
    s = list(es.pdata) if es.pdata is not None else None
    ref = brute.BruteES(name, D, N, sigma, lr, seed, lo, hi, s=s)
    np.testing.assert_array_equal(es.m[0], np.array(ref.m, np.float32))
    for t in range(50):
        es.set_state(np.array([ref.m], np.float32), np.array([ref.m1], np.float32),
                     np.array([ref.v], np.float32), ref.t)
        x_or = es.ask()[0]
        out = es.tell(None)
        r = ref.generation()
        np.testing.assert_array_equal(x_or, np.array(r["X"], np.float32))
        for a, b in zip(out["fitness"][0], r["fitness"]):
            assert _ulps(a, b) <= 1.0, (t, a, b)
        if list(O.ranks(out["fitness"][0])) != brute.ranks(r["fitness"]):
            # only a 1-ulp near-tie may reorder; then shaping legitimately differs
            continue
        np.testing.assert_array_equal(out["y"][0], np.array(r["y"], np.float32))
        E = np.array(r["E"], np.float64)
        scale = np.abs(np.array(r["y"], np.float64)) @ np.abs(E) / (N * np.float32(sigma))
        err = np.abs(out["g"][0].astype(np.float64) - np.array(r["g"], np.float64))
        assert np.all(err <= 2 ** -23 * np.abs(np.array(r["g"])) + 1e-12 * scale + 1e-38), (t, err)
        if np.array_equal(out["g"][0], np.array(r["g"], np.float32)):
            np.testing.assert_array_equal(es.m[0], np.array(ref.m, np.float32))
            np.testing.assert_array_equal(es.m1[0], np.array(ref.m1, np.float32))
            np.testing.assert_array_equal(es.v[0], np.array(ref.v, np.float32))
        else:
            np.testing.assert_allclose(es.m[0], np.array(ref.m, np.float32), rtol=0,
                                       atol=1e-5 * max(lr, float(np.max(np.abs(ref.m)))))


def test_brute_f32_rounding():
    from fractions import Fraction
    assert brute.f32(Fraction(1, 3)) == float(np.float32(1 / 3))
    assert brute.f32(1 + 2 ** -24) == 1.0            # tie -> even
    assert brute.f32(1 + 3 * 2 ** -24) == 1 + 2 ** -22  # tie -> even (up)
    assert brute.f32(2 ** -149) == 2 ** -149           # smallest subnormal
    assert brute.f32(Fraction(2 ** -150)) == 0.0       # tie -> even (zero)
    assert brute.f32(-7.25) == -7.25
    assert math.isinf(brute.f32(2.0 ** 128))
    # fused multiply-add is one rounding: (1+2^-12)^2 - 1 keeps the 2^-24 term
    a = 1 + 2 ** -12
    assert brute.fma32(a, a, -1.0) == 2 ** -11 + 2 ** -24
