"""Pins of the oracle's schedule, per-run hyper-parameter, z-score and
weight-decay additions (App. B schedules; Sec. 2.2 vmap over hyper-parameters;
Sec. 3.2 fitness shaping transformations).

Each property is checked against something other than the oracle itself: the
closed form of the exponential schedule, the exact-rational brute force
(``oracle/brute.py``), scipy's z-score, the sphere problem, and the
sigma-independence of the finite-difference estimate on a linear function."""
import math

import numpy as np
import pytest
import scipy.stats

from oracle import brute
from oracle import oracle as O


def _ulps(a, b):
    a, b = np.float32(a), np.float32(b)
    return abs(float(a) - float(b)) / float(np.spacing(np.float32(max(abs(a), abs(b), 1e-30))))


# ---------------------------------------------------------------------------
# schedules
@pytest.mark.parametrize("x0,rate,final", [(0.1, 0.999, 0.01), (0.05, 0.9, 0.01), (0.02, 0.5, 0.001),
                                           (0.01, 0.999, 0.02), (0.3, 1.0, 0.0)])
def test_schedule_follows_closed_form(x0, rate, final):
    x = np.float32(x0)
    prev = math.inf
    for t in range(1, 3000):
        x = O.decay(float(x), rate, final)
        exact = x0 * rate ** t  # fp64 closed form of the undamped product
        rel = t * 2.0 ** -23
        assert x <= prev or x == np.float32(final)
        prev = x
        if exact * (1 + rel) < final:
            assert x == np.float32(final)
        elif exact * (1 - rel) > final:
            assert abs(x - exact) <= rel * exact + 2 ** -24 * x0, (t, x, exact)
        if rate == 1.0:
            assert x == np.float32(x0) or x == np.float32(final)


def test_schedule_matches_brute_force():
    D, N, T = 3, 6, 40
    kw = dict(sigma_decay=0.95, sigma_final=0.03, lr_decay=0.9, lr_final=0.004)
    cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.1, lr=0.05, seed=9, init=O.INIT_UNIFORM,
                         init_lo=-3.0, init_hi=3.0, problem=O.PROB_SPHERE, **kw)
    es = O.OracleES(cfg)
    ref = brute.BruteES("sphere", D, N, 0.1, 0.05, 9, -3.0, 3.0, **kw)
    for t in range(T):
        es.set_state(np.array([ref.m], np.float32), np.array([ref.m1], np.float32),
                     np.array([ref.v], np.float32), ref.t)
        es.set_hparams([ref.sigma], [ref.lr])
        x = es.ask()[0]
        out = es.tell(None)
        r = ref.generation()
        np.testing.assert_array_equal(x, np.array(r["X"], np.float32))
        assert es.sigma[0] == np.float32(ref.sigma) and es.lr[0] == np.float32(ref.lr), t
        if list(O.ranks(out["fitness"][0])) == brute.ranks(r["fitness"]):
            np.testing.assert_array_equal(out["y"][0], np.array(r["y"], np.float32))
    assert ref.sigma == np.float32(0.03) and ref.lr == np.float32(0.004)


def test_schedule_sigma_used_consistently():
    """Raw shaping on f(x) = a.x: f(m + s e) - f(m - s e) = 2 s a.e, so the
    estimate is (2/N) sum_p (a.e_p) e_p whatever sigma_t is -- it only holds
    if ask and tell use the same decayed sigma."""
    D, N = 16, 64
    a = np.linspace(-1.0, 1.0, D)
    cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.2, lr=0.01, seed=4, init=O.INIT_ZERO,
                         problem=O.PROB_NONE, shaping=O.SHAPE_RAW, sigma_decay=0.5, sigma_final=0.0)
    es = O.OracleES(cfg)
    for t in range(6):
        sig = float(es.sigma[0])
        x = es.ask()[0].astype(np.float64)
        f = (x @ a).astype(np.float32)[None, :]
        out = es.tell(f)
        E = np.stack([O.noise(cfg, 0, t, p) for p in range(N // 2)]).astype(np.float64)
        g_ref = (2.0 / N) * ((E @ a) @ E)
        err = np.max(np.abs(out["g"][0] - g_ref))
        # x is rounded to fp32 around m ~ 1, so a.x carries ~1e-7 |m| of noise
        assert err <= 2e-6 * max(1.0, float(np.max(np.abs(es.m)))) / sig + 1e-5 * np.max(np.abs(g_ref)), (t, err)
        assert sig == np.float32(0.2) * 0.5 ** t


def test_per_run_hyperparameters_equal_standalone_runs():
    R, D, N = 3, 5, 8
    sig = np.array([0.1, 0.05, 0.2], np.float32)
    lr = np.array([0.02, 0.01, 0.005], np.float32)
    base = dict(num_dims=D, popsize=N, seed=21, init=O.INIT_UNIFORM, init_lo=-2.0, init_hi=2.0,
                problem=O.PROB_ROSENBROCK, sigma_decay=0.97, sigma_final=0.04, lr_decay=0.99, lr_final=0.004)
    es = O.OracleES(O.OracleConfig(num_runs=R, **base))
    es.set_hparams(sig, lr)
    es.run(12)
    for r in range(R):
        one = O.OracleES(O.OracleConfig(num_runs=1, **dict(base, seed=21 + r, sigma=float(sig[r]), lr=float(lr[r]))))
        one.run(12)
        np.testing.assert_array_equal(es.m[r], one.m[0])
        assert es.sigma[r] == one.sigma[0] and es.lr[r] == one.lr[0]


# ---------------------------------------------------------------------------
# z-score
def test_zscore_against_scipy_and_invariants():
    rng = np.random.default_rng(3)
    for N in (2, 3, 8, 100, 1001):
        f = (rng.standard_normal(N) * 7 + 3).astype(np.float32)
        y = O.shape_full(f, shaping=O.SHAPE_Z_SCORE)
        k = f.astype(np.float64)
        z = scipy.stats.zscore(k, ddof=0)
        sd = np.std(k)
        np.testing.assert_allclose(y, z * sd / (sd + 1e-10), rtol=2e-7, atol=1e-7)
        assert abs(float(np.sum(y.astype(np.float64)))) <= N * 1.2e-7 * 3
        assert abs(float(np.mean(y.astype(np.float64) ** 2)) - 1.0) <= 1e-6
        # maximisation flips the sign; positive affine maps change nothing
        ym = O.shape_full(f, maximize=1, shaping=O.SHAPE_Z_SCORE)
        np.testing.assert_allclose(ym, -y, atol=2e-7)
        ya = O.shape_full((f.astype(np.float64) * 4.0 - 1.0).astype(np.float32), shaping=O.SHAPE_Z_SCORE)
        np.testing.assert_allclose(ya, y, rtol=1e-5, atol=1e-5)


def test_zscore_nonfinite_members_get_zero():
    f = np.array([1.0, np.nan, 3.0, np.inf, -2.0, -np.inf, 5.0], np.float32)
    y = O.shape_full(f, shaping=O.SHAPE_Z_SCORE)
    fin = np.isfinite(f)
    assert np.all(y[~fin] == 0.0)
    k = f[fin].astype(np.float64)
    np.testing.assert_allclose(y[fin], (k - k.mean()) / (k.std() + 1e-10), rtol=2e-7, atol=1e-7)
    assert np.all(O.shape_full(np.full(5, 2.5, np.float32), shaping=O.SHAPE_Z_SCORE) == 0.0)


def test_zscore_matches_exact_rational():
    rng = np.random.default_rng(11)
    for _ in range(20):
        N = int(rng.integers(2, 9))
        f = (rng.standard_normal(N) * 10).astype(np.float32)
        y = O.shape_full(f, shaping=O.SHAPE_Z_SCORE)
        yb = brute.zscore([float(v) for v in f])
        for a, b in zip(y, yb):
            assert _ulps(a, b) <= 1.0, (f, a, b)


# ---------------------------------------------------------------------------
# weight decay
def test_penalty_is_sphere_over_d():
    cfg = O.OracleConfig(num_dims=37, popsize=10, seed=5, init=O.INIT_UNIFORM, init_lo=-2.0, init_hi=2.0)
    m = O.init_mean(cfg, 0)
    pen = O.penalty(cfg, 0, 3, m)
    X = O.population(cfg, 0, 3, m)
    for j in range(cfg.popsize):
        sph = O.fitness_bbob(O.PROB_SPHERE, X[j])
        assert _ulps(pen[j], np.float32(sph) / np.float32(37)) <= 1.0
        assert _ulps(pen[j], np.mean(X[j].astype(np.float64) ** 2)) <= 0.5


def test_weight_decay_keys_match_exact_rounding():
    rng = np.random.default_rng(8)
    for maximize in (0, 1):
        f = (rng.standard_normal(64) * 3).astype(np.float32)
        f[5], f[9] = np.nan, np.inf
        pen = np.abs(rng.standard_normal(64) * 2).astype(np.float32)
        w = np.float32(0.37)
        keys = [O._lib.or_shaped_key(float(f[j]), float(pen[j]), maximize, float(w)) if O._lib else None
                for j in range(64)]
        ref = brute.shaped_keys([float(v) for v in f], [float(v) for v in pen], maximize, float(w))
        for a, b in zip(keys, ref):
            assert (math.isinf(a) and a == b) or np.float32(a) == np.float32(b), (a, b)
        y = O.shape_full(f, pen, maximize=maximize, shaping=O.SHAPE_RAW, w_decay=float(w))
        for a, b in zip(y, ref):
            assert (math.isinf(a) and a == b) or np.float32(a) == np.float32(b)


def test_weight_decay_breaks_fitness_ties_by_size():
    f = np.zeros(8, np.float32)
    pen = np.array([3.0, 1.0, 2.0, 0.5, 4.0, 0.25, 8.0, 6.0], np.float32)
    y = O.shape_full(f, pen, shaping=O.SHAPE_CENTERED_RANK, w_decay=0.1)
    order = np.argsort(pen, kind="stable")
    assert list(np.argsort(y, kind="stable")) == list(order)
    for shaping in (O.SHAPE_CENTERED_RANK, O.SHAPE_Z_SCORE, O.SHAPE_RAW):
        g = (np.arange(8) % 3).astype(np.float32)
        np.testing.assert_array_equal(O.shape_full(g, pen, shaping=shaping, w_decay=0.0),
                                      O.shape_full(g, None, shaping=shaping))
    np.testing.assert_array_equal(O.shape_full(g, None, shaping=O.SHAPE_CENTERED_RANK), O.shape(g))


def test_weight_decay_pulls_mean_towards_zero():
    """Flat fitness plus weight decay: the strategy minimises the mean square."""
    cfg = O.OracleConfig(num_dims=20, popsize=32, sigma=0.1, lr=0.05, seed=2, init=O.INIT_UNIFORM,
                         init_lo=1.0, init_hi=2.0, problem=O.PROB_NONE, w_decay=1.0)
    es = O.OracleES(cfg)
    n0 = float(np.mean(es.m ** 2))
    for _ in range(40):
        es.tell(np.zeros((1, 32), np.float32))
    assert float(np.mean(es.m ** 2)) < 0.5 * n0


@pytest.mark.parametrize("shaping", ["centered", "zscore"])
def test_weight_decay_and_zscore_generation_match_brute(shaping):
    D, N = 3, 6
    kw = dict(w_decay=0.5)
    code = {"centered": O.SHAPE_CENTERED_RANK, "zscore": O.SHAPE_Z_SCORE}[shaping]
    cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.1, lr=0.05, seed=13, init=O.INIT_UNIFORM,
                         init_lo=-2.0, init_hi=2.0, problem=O.PROB_RASTRIGIN, shaping=code, **kw)
    es = O.OracleES(cfg)
    ref = brute.BruteES("rastrigin", D, N, 0.1, 0.05, 13, -2.0, 2.0, shaping=shaping, **kw)
    for t in range(25):
        es.set_state(np.array([ref.m], np.float32), np.array([ref.m1], np.float32),
                     np.array([ref.v], np.float32), ref.t)
        out = es.tell(None)
        r = ref.generation()
        for a, b in zip(out["fitness"][0], r["fitness"]):
            assert _ulps(a, b) <= 1.0
        if not all(_ulps(a, b) == 0 for a, b in zip(out["fitness"][0], r["fitness"])):
            continue  # a 1-ulp fitness difference may legitimately reorder a near-tie
        for a, b in zip(out["y"][0], r["y"]):
            assert _ulps(a, b) <= 1.0, (t, a, b)
