"""Pins of the oracle's Sep-CMA-ES (Ros & Hansen 2008; Table 1 EOD row, App. B
table: sigma init and elite ratio): the exact-rational brute force, the
recombination weights' closed forms, invariance of the trajectory under a
monotone transform of the fitness (selection uses ranks only), and the
textbook linear convergence on the sphere."""
import math

import numpy as np
import pytest

from oracle import brute
from oracle import oracle as O


def _cfg(**kw):
    base = dict(num_dims=5, popsize=8, sigma=0.5, seed=7, init=O.INIT_UNIFORM, init_lo=-3.0, init_hi=3.0,
                problem=O.PROB_SPHERE, strategy=O.STRAT_SEP_CMA, elite_ratio=0.5)
    base.update(kw)
    return O.OracleConfig(**base)


@pytest.mark.parametrize("N,ratio", [(8, 0.5), (16, 0.2), (10, 0.4), (64, 0.5), (5, 0.1)])
def test_weights_closed_form(N, ratio):
    w = O.cma_weights(_cfg(popsize=N, elite_ratio=ratio))
    mu = max(1, int(math.floor(ratio * N)))
    assert len(w) == mu
    assert abs(w.sum() - 1.0) <= 1e-15 * mu and np.all(w > 0) and np.all(np.diff(w) < 0)
    if mu > 1:
        assert abs(w[0] / w[-1] - math.log(mu + 0.5) / math.log((mu + 0.5) / mu)) <= 1e-12 * w[0] / w[-1]
    mu_eff = 1.0 / np.sum(w ** 2)
    assert 1.0 <= mu_eff <= mu + 1e-12


@pytest.mark.parametrize("problem,name", [(O.PROB_SPHERE, "sphere"), (O.PROB_ROSENBROCK, "rosenbrock")])
@pytest.mark.parametrize("D,N,ratio", [(2, 4, 0.5), (3, 8, 0.5), (4, 6, 0.4)])
def test_sepcma_matches_brute_force(problem, name, D, N, ratio):
    cfg = _cfg(num_dims=D, popsize=N, elite_ratio=ratio, problem=problem, init_lo=-2.0, init_hi=2.0)
    es = O.OracleES(cfg)
    ref = brute.BruteSepCMA(name, D, N, 0.5, 7, -2.0, 2.0, elite_ratio=ratio)
    np.testing.assert_array_equal(es.m[0], np.array(ref.m, np.float32))
    for t in range(30):
        es.set_state(np.array([ref.m], np.float32), np.array([ref.ps], np.float32), np.array([ref.pc], np.float32),
                     ref.t, sig=np.array([ref.C], np.float32))
        es.sigma[0] = np.float32(ref.sigma)
        x = es.ask()[0]
        out = es.tell(None)
        r = ref.generation()
        np.testing.assert_array_equal(x, np.array(r["X"], np.float32))
        if list(O.ranks(out["fitness"][0])) != brute.ranks(r["fitness"]):
            continue
        for a, b in ((es.m[0], ref.m), (es.m1[0], ref.ps), (es.v[0], ref.pc), (es.sig[0], ref.C)):
            b = np.array(b, np.float64)
            assert np.all(np.abs(a - b) <= 1e-6 * np.maximum(np.abs(b), 1e-3)), (t, a, b)
        assert abs(float(es.sigma[0]) - ref.sigma) <= 1e-6 * ref.sigma


def test_sepcma_invariant_to_monotone_fitness_transform():
    cfg = _cfg(num_dims=6, popsize=12, problem=O.PROB_NONE)
    a, b = O.OracleES(cfg), O.OracleES(cfg)
    for _ in range(20):
        x = a.ask()[0].astype(np.float64)
        f = np.sum((x - 0.3) ** 2, axis=1)
        a.tell(f.astype(np.float32)[None])
        b.tell(np.exp(np.sqrt(f)).astype(np.float32)[None])  # strictly increasing in f
        np.testing.assert_array_equal(a.m, b.m)
        np.testing.assert_array_equal(a.sig, b.sig)
        np.testing.assert_array_equal(a.sigma, b.sigma)


def test_sepcma_converges_linearly_on_the_sphere():
    cfg = _cfg(num_dims=10, popsize=16, sigma=0.5, init_lo=-3.0, init_hi=3.0)
    es = O.OracleES(cfg)
    f0 = float(np.min(es.eval()))
    logs = []
    for t in range(200):
        out = es.step()
        logs.append(math.log10(max(float(np.min(out["fitness"])), 1e-300)))
    assert logs[-1] < math.log10(f0) - 12
    # roughly constant progress per generation (linear convergence)
    slope1 = (logs[99] - logs[49]) / 50
    slope2 = (logs[199] - logs[149]) / 50
    assert slope1 < -0.02 and slope2 < -0.02
