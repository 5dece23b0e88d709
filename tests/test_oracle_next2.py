"""Pins of the oracle's PGPE, SNES and ClipUp additions (Table 1 strategies
PGPE and SNES, the ClipUp optimiser of Sec. 3.1, App. B hyper-parameter
tables): the exact-rational brute force on tiny problems, closed forms
(softmax utility ratios, ClipUp's geometric velocity, the clipped sigma
step, E[g] = a * sigma^2 for PGPE on a linear function) and the expected
direction of the sigma updates."""
import math

import numpy as np
import pytest

from oracle import brute
from oracle import oracle as O


def _ulps(a, b):
    a, b = np.asarray(a, np.float32), np.asarray(b, np.float32)
    scale = np.spacing(np.maximum(np.maximum(np.abs(a), np.abs(b)), np.float32(1e-30)))
    return np.abs(a.astype(np.float64) - b.astype(np.float64)) / scale


CASES = [("pgpe", O.STRAT_PGPE, "adam"), ("pgpe", O.STRAT_PGPE, "clipup"), ("snes", O.STRAT_SNES, "adam"),
         ("openai", O.STRAT_OPENAI_ES, "clipup")]


@pytest.mark.parametrize("name,code,opt", CASES)
@pytest.mark.parametrize("D,N", [(1, 4), (3, 6), (4, 8)])
def test_family_matches_brute_force(name, code, opt, D, N):
    lr = 1.0 if name == "snes" else 0.05
    kw = dict(sigma_lr=0.2 if name == "pgpe" else 0.3, max_change=0.2, optimizer=opt, max_speed=0.1,
              momentum=0.9, beta=12.0)
    ref = brute.BruteFamily(name, "sphere", D, N, 0.3, lr, 40 + D, -2.0, 2.0, **kw)
    cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.3, lr=lr, seed=40 + D, init=O.INIT_UNIFORM, init_lo=-2.0,
                         init_hi=2.0, problem=O.PROB_SPHERE, strategy=code,
                         optimizer=O.OPT_CLIPUP if opt == "clipup" else O.OPT_ADAM, sigma_lr=kw["sigma_lr"],
                         sigma_max_change=0.2, clipup_max_speed=0.1, clipup_momentum=0.9, snes_temperature=12.0)
    es = O.OracleES(cfg)
    np.testing.assert_array_equal(es.m[0], np.array(ref.m, np.float32))
    for t in range(25):
        es.set_state(np.array([ref.m], np.float32), np.array([ref.m1], np.float32), np.array([ref.v], np.float32),
                     ref.t, sig=np.array([ref.sig], np.float32), vel=np.array([ref.vel], np.float32))
        if name == "openai":
            es.sigma[0] = np.float32(ref.sig[0])
        x = es.ask()[0]
        out = es.tell(None)
        r = ref.generation()
        np.testing.assert_array_equal(x, np.array(r["X"], np.float32))
        for a, b in zip(out["fitness"][0], r["fitness"]):
            assert _ulps(a, b) <= 1.0
        if list(O.ranks(out["fitness"][0])) != brute.ranks(r["fitness"]):
            continue  # a 1-ulp near-tie may reorder
        tol = 1e-6 * max(float(np.max(np.abs(ref.m))), lr) + 1e-12
        assert np.max(np.abs(es.m[0] - np.array(ref.m, np.float32))) <= tol, (t, es.m[0], ref.m)
        if name != "openai":
            assert np.all(_ulps(es.sig[0], np.array(ref.sig, np.float32)) <= 2.0), (t, es.sig[0], ref.sig)
        if opt == "clipup":
            assert np.max(np.abs(es.vel[0] - np.array(ref.vel, np.float32))) <= 1e-6 * 0.1 + 1e-12


# ---------------------------------------------------------------------------
# PGPE
def test_pgpe_flat_fitness_moves_nothing():
    cfg = O.OracleConfig(num_dims=9, popsize=10, sigma=0.2, lr=0.05, seed=1, problem=O.PROB_NONE,
                         strategy=O.STRAT_PGPE, shaping=O.SHAPE_RAW)
    es = O.OracleES(cfg)
    m0, s0 = es.m.copy(), es.sig.copy()
    for _ in range(3):
        es.tell(np.full((1, 10), 3.5, np.float32))
    np.testing.assert_array_equal(es.m, m0)
    np.testing.assert_array_equal(es.sig, s0)


def test_pgpe_mean_gradient_expectation_on_linear_function():
    """Raw shaping on f = a.x: a_p = y+ - y- = 2 sum_k a_k sigma_k z_pk, so
    E[g_d] = E[sigma_d A_d / N] = a_d sigma_d^2."""
    D, N, S = 6, 64, 300
    a = np.array([1.0, -2.0, 0.5, 0.0, 3.0, -1.0])
    sig = np.array([0.1, 0.2, 0.3, 0.05, 0.15, 0.25], np.float32)
    acc = np.zeros(D)
    acc2 = np.zeros(D)
    for seed in range(S):
        cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.1, lr=0.0, seed=seed, init=O.INIT_ZERO,
                             problem=O.PROB_NONE, strategy=O.STRAT_PGPE, shaping=O.SHAPE_RAW, sigma_lr=0.0)
        es = O.OracleES(cfg)
        es.sig[0] = sig
        x = es.ask()[0].astype(np.float64)
        out = es.tell((x @ a).astype(np.float32)[None])
        acc += out["g"][0]
        acc2 += out["g"][0].astype(np.float64) ** 2
    mean = acc / S
    sd = np.sqrt(np.maximum(acc2 / S - mean ** 2, 0) / S)
    expect = a * sig.astype(np.float64) ** 2
    assert np.all(np.abs(mean - expect) <= 5 * sd + 1e-9), (mean, expect, sd)


def test_pgpe_sigma_step_is_clipped_to_max_change():
    cfg = O.OracleConfig(num_dims=16, popsize=32, sigma=0.2, lr=0.01, seed=3, init=O.INIT_ZERO,
                         problem=O.PROB_SPHERE, strategy=O.STRAT_PGPE, sigma_lr=1e6, sigma_max_change=0.2)
    es = O.OracleES(cfg)
    s0 = es.sig[0].copy()
    es.step()
    lim = (np.float32(0.2) * s0).astype(np.float32)
    up, dn = (s0 + lim).astype(np.float32), (s0 - lim).astype(np.float32)
    assert np.all((es.sig[0] == up) | (es.sig[0] == dn))


def test_pgpe_sigma_shrinks_at_the_optimum():
    """At the sphere's optimum the best members are the small perturbations:
    the sigma gradient is positive on average and sigma decreases."""
    ratios = []
    for seed in range(40):
        cfg = O.OracleConfig(num_dims=8, popsize=32, sigma=0.5, lr=0.0, seed=seed, init=O.INIT_ZERO,
                             problem=O.PROB_SPHERE, strategy=O.STRAT_PGPE, sigma_lr=0.2)
        es = O.OracleES(cfg)
        es.step()
        ratios.append(float(np.mean(es.sig[0])) / 0.5)
    assert np.mean(ratios) < 0.99 and max(ratios) < 1.0


# ---------------------------------------------------------------------------
# SNES
@pytest.mark.parametrize("N,beta", [(8, 12.0), (256, 16.0), (64, 0.0), (1024, 32.0)])
def test_snes_table_closed_form(N, beta):
    w = O.snes_table(N, beta).astype(np.float64)
    assert abs(w.sum() - 1.0) <= N * 2 ** -24
    assert np.all(np.diff(w) >= 0)
    r = w[1:] / w[:-1]
    assert np.all(np.abs(r - math.exp(beta / N)) <= 4 * 2 ** -24 * math.exp(beta / N))
    if beta == 0.0:
        assert np.all(w == np.float32(1.0 / N))


def test_snes_moves_downhill_and_expands_sigma_on_a_slope():
    D, N = 10, 32
    a = np.linspace(-1.0, 1.0, D)
    cos, grow = [], []
    for seed in range(30):
        cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.3, lr=1.0, seed=seed, init=O.INIT_ZERO,
                             problem=O.PROB_NONE, strategy=O.STRAT_SNES, sigma_lr=0.2, snes_temperature=12.0)
        es = O.OracleES(cfg)
        x = es.ask()[0].astype(np.float64)
        es.tell((x @ a).astype(np.float32)[None])
        dm = es.m[0].astype(np.float64)
        cos.append(dm @ -a / (np.linalg.norm(dm) * np.linalg.norm(a)))
        grow.append(np.mean(np.log(es.sig[0] / 0.3)))
    assert np.mean(cos) > 0.5
    assert np.mean(grow) > 0.0


def test_snes_sigma_shrinks_at_the_optimum():
    logs = []
    for seed in range(30):
        cfg = O.OracleConfig(num_dims=8, popsize=32, sigma=0.5, lr=0.0, seed=seed, init=O.INIT_ZERO,
                             problem=O.PROB_SPHERE, strategy=O.STRAT_SNES, sigma_lr=0.3, snes_temperature=12.0)
        es = O.OracleES(cfg)
        es.step()
        logs.append(np.mean(np.log(es.sig[0] / 0.5)))
    assert np.mean(logs) < 0.0


# ---------------------------------------------------------------------------
# ClipUp
def test_clipup_first_step_and_geometric_velocity():
    cfg = O.OracleConfig(num_dims=50, popsize=4, clipup_max_speed=0.3, clipup_momentum=0.9)
    rng = np.random.default_rng(5)
    g = rng.standard_normal(50).astype(np.float32)
    m = np.zeros(50, np.float32)
    vel = np.zeros(50, np.float32)
    lr = 0.05
    for k in range(1, 40):
        m_new, vel = O.clipup(cfg, lr, g, m, vel)
        speed = float(np.linalg.norm(vel.astype(np.float64)))
        expect = min(lr * (1 - 0.9 ** k) / (1 - 0.9), 0.3)
        assert abs(speed - expect) <= 1e-5 * expect, (k, speed, expect)
        cosang = float(vel.astype(np.float64) @ g / (speed * np.linalg.norm(g.astype(np.float64))))
        assert cosang > 1 - 1e-6
        np.testing.assert_array_equal(m_new, (m - vel).astype(np.float32))
        m = m_new
    # zero gradient: no step beyond the decaying velocity
    m2, v2 = O.clipup(cfg, lr, np.zeros(50, np.float32), m, vel)
    np.testing.assert_array_equal(v2, (np.float32(0.9) * vel).astype(np.float32))
