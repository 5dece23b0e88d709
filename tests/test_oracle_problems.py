"""Pins of the oracle's benchmark problems (BBOB family, Sec. 3.2): optima and
closed-form values that do not depend on retyping the formula."""
import math

import numpy as np
import pytest

from oracle import brute
from oracle import oracle as O


@pytest.mark.parametrize("D", [1, 2, 16, 100, 1000])
def test_optima_are_zero(D):
    z = np.zeros(D, np.float32)
    one = np.ones(D, np.float32)
    assert O.fitness_bbob(O.PROB_SPHERE, z) == 0.0
    assert O.fitness_bbob(O.PROB_ROSENBROCK, one) == 0.0
    assert O.fitness_bbob(O.PROB_RASTRIGIN, z, a=10.0) == 0.0
    s = O.normals(2, O.DOM_PROBLEM, 0, 0, 0, D)
    assert O.fitness_bbob(O.PROB_SHIFTED_SPHERE, s, s) == 0.0


@pytest.mark.parametrize("D", [1, 3, 16, 1000])
def test_closed_forms(D):
    z = np.zeros(D, np.float32)
    one = np.ones(D, np.float32)
    half = np.full(D, 0.5, np.float32)
    assert O.fitness_bbob(O.PROB_SPHERE, one) == D
    assert O.fitness_bbob(O.PROB_SPHERE, -2 * one) == 4 * D
    # Rosenbrock at 0: each of the D-1 terms is (1-0)^2 = 1
    assert O.fitness_bbob(O.PROB_ROSENBROCK, z) == D - 1
    # at -1: 100*(-1-1)^2 + (1+1)^2 = 404 per term
    assert O.fitness_bbob(O.PROB_ROSENBROCK, -one) == 404 * (D - 1)
    # Rastrigin at 1/2: x^2 - A cos(pi) = 1/4 + A per coordinate
    assert O.fitness_bbob(O.PROB_RASTRIGIN, half, a=10.0) == pytest.approx(10 * D + D * 10.25, rel=1e-7)
    # at integers, cos(2 pi k) = 1: f = sum k^2
    ks = (np.arange(D) % 5 - 2).astype(np.float32)
    assert O.fitness_bbob(O.PROB_RASTRIGIN, ks, a=10.0) == pytest.approx(float(np.sum(ks.astype(np.float64) ** 2)), abs=1e-9 * D)
    s = O.normals(2, O.DOM_PROBLEM, 0, 0, 0, D)
    assert O.fitness_bbob(O.PROB_SHIFTED_SPHERE, s + 1, s) == pytest.approx(D, rel=1e-6)


def test_rosenbrock_is_the_only_neighbour_coupled_problem():
    # permuting coordinates leaves sphere and Rastrigin unchanged, not Rosenbrock
    rng = np.random.default_rng(3)
    x = rng.normal(size=12).astype(np.float32)
    p = x[::-1].copy()
    assert O.fitness_bbob(O.PROB_SPHERE, x) == pytest.approx(O.fitness_bbob(O.PROB_SPHERE, p), rel=1e-7)
    assert O.fitness_bbob(O.PROB_RASTRIGIN, x) == pytest.approx(O.fitness_bbob(O.PROB_RASTRIGIN, p), rel=1e-7)
    assert O.fitness_bbob(O.PROB_ROSENBROCK, x) != pytest.approx(O.fitness_bbob(O.PROB_ROSENBROCK, p), rel=1e-3)


@pytest.mark.parametrize("prob,name", [(O.PROB_SPHERE, "sphere"), (O.PROB_ROSENBROCK, "rosenbrock"),
                                       (O.PROB_RASTRIGIN, "rastrigin"), (O.PROB_SHIFTED_SPHERE, "shifted_sphere")])
def test_problems_match_brute(prob, name):
    rng = np.random.default_rng(prob)
    for D in (1, 2, 3, 4, 9):
        x = (rng.normal(size=D) * 2).astype(np.float32)
        s = rng.normal(size=D).astype(np.float32)
        got = O.fitness_bbob(prob, x, s)
        want = brute.fitness(name, list(x), list(s))
        # fp64 sequential sum vs exact sum: at most one fp32 ulp apart
        assert abs(got - want) <= float(np.spacing(np.float32(abs(want)))), (D, got, want)
