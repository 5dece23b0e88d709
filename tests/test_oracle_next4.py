"""Pins of the oracle's Sep-CMA-ES (Ros & Hansen 2008; Table 1 EOD row, App. B
table: sigma init and elite ratio): the exact-rational brute force, the
recombination weights' closed forms, invariance of the trajectory under a
monotone transform of the fitness (selection uses ranks only), the textbook
linear convergence on the sphere, and -- under random selection -- the
expectations the adaptation settings are built to meet (stationary paths,
unbiased covariance with and without the stall of p_c, zero log-step drift),
from which the rates c_s, c_c, c1, c_mu, the damping d_s, chi_D and the stall
threshold are read back and compared with the published settings."""
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


# --------------------------------------------------------------------------
# Random selection: fitness drawn independently of the population, so the mu
# elites are a uniformly random subset of N independent members.  Then the
# weighted elite step zw_d = sum_i w_i z_{e_i,d} is N(0, 1/mu_eff) in every
# coordinate and q_d = sum_i w_i z_{e_i,d}^2 has mean sum_i w_i = 1 and
# variance 2/mu_eff.  These facts fix what the adaptation must do in
# expectation (Hansen, "The CMA Evolution Strategy: A Tutorial", 2016: the
# normalisations of the paths are chosen so that, under random selection,
# p_sigma ~ N(0, I), p_c ~ N(0, C), E[C'] = C and E[log sigma'] = 0 up to the
# chi_D approximation).  Each run of an R-batch has its own Philox key, so the
# R runs are independent samples.  The settings the extracted rates are
# compared with are the tutorial's defaults (its Table 1) with the separable
# factor (D + 2)/3 of Ros & Hansen (2008) on c1 and c_mu.
# --------------------------------------------------------------------------
def _tutorial_settings(D, mu_eff):
    c_s = (mu_eff + 2.0) / (D + mu_eff + 5.0)
    d_s = 1.0 + 2.0 * max(0.0, math.sqrt((mu_eff - 1.0) / (D + 1.0)) - 1.0) + c_s
    c_c = (4.0 + mu_eff / D) / (D + 4.0 + 2.0 * mu_eff / D)
    c1 = 2.0 / ((D + 1.3) ** 2 + mu_eff)
    cmu = min(1.0 - c1, 2.0 * (mu_eff - 2.0 + 1.0 / mu_eff) / ((D + 2.0) ** 2 + mu_eff))
    sep = (D + 2.0) / 3.0
    c1s = min(1.0, c1 * sep)
    return dict(c_s=c_s, d_s=d_s, c_c=c_c, c1=c1s, cmu=min(1.0 - c1s, cmu * sep))


def _chi_mean(D):
    """E|N(0, I_D)| = sqrt(2) Gamma((D+1)/2) / Gamma(D/2), exactly."""
    return math.sqrt(2.0) * math.exp(math.lgamma((D + 1) / 2.0) - math.lgamma(D / 2.0))


def _random_selection_tell(D, N, R, ps, pc, C, t, seed, fseed):
    """One Sep-CMA-ES tell of R independent runs from the given state with
    fitness independent of the population; returns (p_sigma', p_c', C',
    sigma' / sigma, m' - m) as float64 arrays."""
    cfg = _cfg(num_dims=D, popsize=N, num_runs=R, sigma=1.0, seed=seed, problem=O.PROB_NONE, elite_ratio=0.5)
    es = O.OracleES(cfg)
    m0 = np.zeros((R, D), np.float32)
    es.set_state(m0, ps.astype(np.float32), pc.astype(np.float32), t, sig=C.astype(np.float32))
    es.sigma[:] = 1.0
    f = np.random.default_rng(fseed).normal(size=(R, N)).astype(np.float32)
    es.tell(f)
    return (es.m1.astype(np.float64), es.v.astype(np.float64), es.sig.astype(np.float64),
            es.sigma.astype(np.float64), es.m.astype(np.float64))


SEL_D, SEL_N, SEL_R = 16, 16, 10000


@pytest.fixture(scope="module")
def sel():
    D, N, R = SEL_D, SEL_N, SEL_R
    w = O.cma_weights(_cfg(num_dims=D, popsize=N, elite_ratio=0.5))
    mu_eff = 1.0 / float(np.sum(w ** 2))
    rng = np.random.default_rng(2024)
    C = rng.uniform(0.5, 2.0, size=(R, D))
    ps = rng.normal(size=(R, D))                   # stationary p_sigma ~ N(0, I)
    pc = rng.normal(size=(R, D)) * np.sqrt(C)      # stationary p_c ~ N(0, C)
    ps32, pc32, C32 = (a.astype(np.float32).astype(np.float64) for a in (ps, pc, C))
    # batch A: stationary paths, h = 1 (|p_sigma'| stays far below the threshold)
    A = _random_selection_tell(D, N, R, ps32, pc32, C32, 1000, seed=100, fseed=1)
    # batch B: the same keys and fitness, p_sigma far beyond the threshold (h = 0)
    B = _random_selection_tell(D, N, R, np.full((R, D), 50.0), pc32, C32, 1000, seed=100, fseed=1)
    # batch Z: p_c = 0, h = 0, C = 1 (c1 and c_mu from the first two moments of C')
    Z = _random_selection_tell(D, N, R, np.full((R, D), 50.0), np.zeros((R, D)), np.ones((R, D)), 1000,
                               seed=300, fseed=3)
    return dict(D=D, N=N, R=R, mu_eff=mu_eff, ps=ps32, pc=pc32, C=C32, A=A, B=B, Z=Z,
                ref=_tutorial_settings(D, mu_eff))


def _slope(x, y):
    x, y = x.ravel(), y.ravel()
    return float(np.dot(x, y) / np.dot(x, x))


def test_random_selection_p_sigma_stays_standard_normal(sel):
    """p_sigma' = (1 - c_s) p_sigma + sqrt(c_s (2 - c_s) mu_eff) zw keeps
    N(0, I): per-coordinate mean 0, variance 1; the regression slope on the
    previous path is 1 - c_s and the innovation has variance c_s (2 - c_s)."""
    ps1 = sel["A"][0]
    n = ps1.size
    assert abs(ps1.mean()) <= 5.0 / math.sqrt(n)
    assert abs(ps1.var() - 1.0) <= 5.0 * math.sqrt(2.0 / n)
    c_s = sel["ref"]["c_s"]
    b = _slope(sel["ps"], ps1)
    assert abs((1.0 - b) - c_s) <= 5.0 * math.sqrt(c_s * (2 - c_s) / np.sum(sel["ps"] ** 2)), (1 - b, c_s)
    innov = ps1 - (1.0 - c_s) * sel["ps"]
    assert abs(innov.var() / (c_s * (2.0 - c_s)) - 1.0) <= 5.0 * math.sqrt(2.0 / n)


def test_random_selection_p_c_tracks_the_covariance(sel):
    """With h = 1, p_c' = (1 - c_c) p_c + sqrt(c_c (2 - c_c) mu_eff) sqrt(C) zw:
    from p_c ~ N(0, C) it stays N(0, C) (E[p_c'^2 / C] = 1), the slope on p_c is
    1 - c_c, and the innovation has variance c_c (2 - c_c) C."""
    pc1, C = sel["A"][1], sel["C"]
    n = pc1.size
    u = pc1 / np.sqrt(C)
    assert abs(u.mean()) <= 5.0 / math.sqrt(n)
    assert abs(np.mean(u * u) - 1.0) <= 5.0 * math.sqrt(2.0 / n)
    c_c = sel["ref"]["c_c"]
    b = _slope(sel["pc"] / np.sqrt(C), u)
    assert abs((1.0 - b) - c_c) <= 5.0 * math.sqrt(c_c * (2 - c_c) / np.sum(sel["pc"] ** 2 / C)), (1 - b, c_c)
    innov = (pc1 - (1.0 - c_c) * sel["pc"]) / np.sqrt(C)
    assert abs(np.mean(innov ** 2) / (c_c * (2.0 - c_c)) - 1.0) <= 5.0 * math.sqrt(2.0 / n)


def test_random_selection_keeps_the_covariance_unbiased(sel):
    """From stationary paths, E[C'_d / C_d] = 1: the rank-one term gets
    E[p_c'^2] = C and the rank-mu term E[q] = 1, so the rates cancel with the
    (1 - c1 - c_mu) decay whatever their values."""
    r = sel["A"][2] / sel["C"]
    n = r.size
    assert abs(r.mean() - 1.0) <= 5.0 * r.std() / math.sqrt(n), r.mean()


def test_stalled_path_keeps_the_covariance_unbiased(sel):
    """h = 0 stops the p_c increment; the (1 - h) c_c (2 - c_c) C term puts its
    expected square back, so E[C'] does not depend on h.  Batches A (h = 1)
    and B (h = 0) share keys and fitness, hence noise and elites: the paired
    difference of C' has mean 0, and B's p_c only decays, by 1 - c_c."""
    dA, dB = sel["A"][2], sel["B"][2]
    diff = (dA - dB) / sel["C"]
    n = diff.size
    assert abs(diff.mean()) <= 5.0 * diff.std() / math.sqrt(n), diff.mean()
    c_c = sel["ref"]["c_c"]
    np.testing.assert_allclose(sel["B"][1], (1.0 - c_c) * sel["pc"], rtol=1e-6, atol=1e-6)
    # and the paths really differ between the batches (h = 1 in A)
    assert np.max(np.abs(sel["A"][1] - sel["B"][1])) > 0.1


def test_covariance_rates_are_the_separable_settings(sel):
    """Batch Z (p_c = 0, h = 0, C = 1): C' = 1 - c1 (1 - c_c)^2 + c_mu (q - 1),
    so the mean of C' gives c1 and its variance 2 c_mu^2 / mu_eff gives c_mu.
    Both must be the tutorial's rates times (D + 2)/3 (Ros & Hansen 2008)."""
    C1 = sel["Z"][2]
    n = C1.size
    ref = sel["ref"]
    c_c, mu_eff = ref["c_c"], sel["mu_eff"]
    cmu_hat = math.sqrt(C1.var() * mu_eff / 2.0)
    # q is a weighted sum of mu squared normals: its 4th central moment sets the
    # standard error of the variance estimate (computed from the sample)
    k4 = float(np.mean((C1 - C1.mean()) ** 4))
    se_var = math.sqrt(max(k4 - C1.var() ** 2, 0.0) / n)
    assert abs(cmu_hat - ref["cmu"]) <= 5.0 * cmu_hat * 0.5 * se_var / C1.var(), (cmu_hat, ref["cmu"])
    c1_hat = (1.0 - C1.mean()) / (1.0 - c_c) ** 2
    se_c1 = C1.std() / math.sqrt(n) / (1.0 - c_c) ** 2
    assert abs(c1_hat - ref["c1"]) <= 5.0 * se_c1, (c1_hat, ref["c1"])
    # the plain (non-separable) rates are far outside these bounds
    sep = (SEL_D + 2.0) / 3.0
    assert abs(c1_hat - ref["c1"] / sep) > 20 * se_c1


def test_step_size_follows_the_path_length(sel):
    """log(sigma'/sigma) = (c_s / d_s)(|p_sigma'| / chi_D - 1) exactly, so a
    line through (|p_sigma'|, log(sigma'/sigma)) gives chi_D and d_s: chi_D must
    be E|N(0, I)| (the tutorial's series is within 5e-5 of it at D = 16), d_s
    the tutorial damping, and under random selection the mean log-step is 0
    up to that small difference."""
    ps1, sig1 = sel["A"][0], sel["A"][3]
    L = np.linalg.norm(ps1, axis=1)
    z = np.log(sig1)
    slope, icpt = np.polyfit(L, z, 1)
    chi = -icpt / slope
    k = -icpt
    assert abs(chi / _chi_mean(SEL_D) - 1.0) <= 1e-3, (chi, _chi_mean(SEL_D))
    assert abs(sel["ref"]["c_s"] / k - sel["ref"]["d_s"]) <= 1e-4 * sel["ref"]["d_s"]
    assert np.max(np.abs(z - (slope * L + icpt))) <= 1e-6
    assert abs(z.mean()) <= 5.0 * z.std() / math.sqrt(z.size)


@pytest.mark.parametrize("t", [0, 4])
def test_stall_threshold(t):
    """h = 1 exactly when |p_sigma'| / sqrt(1 - (1 - c_s)^(2(t+1))) is below
    (1.4 + 2/(D+1)) E|N(0, I)| (the tutorial's h_sigma); with p_c = 0 a stalled
    path stays exactly 0.  Paths are scaled to straddle the threshold."""
    D, N, R = 8, 16, 400
    w = O.cma_weights(_cfg(num_dims=D, popsize=N, elite_ratio=0.5))
    ref = _tutorial_settings(D, 1.0 / float(np.sum(w ** 2)))
    thr = (1.4 + 2.0 / (D + 1)) * _chi_mean(D) * math.sqrt(1.0 - (1.0 - ref["c_s"]) ** (2 * (t + 1)))
    rng = np.random.default_rng(77 + t)
    u = rng.normal(size=(R, D))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    ps = u * (thr * rng.uniform(0.6, 1.4, size=(R, 1)) / (1.0 - ref["c_s"]))
    ps1, pc1 = _random_selection_tell(D, N, R, ps, np.zeros((R, D)), np.ones((R, D)), t, seed=5, fseed=6)[:2]
    L = np.linalg.norm(ps1, axis=1)
    stalled = np.all(pc1 == 0.0, axis=1)
    assert 50 < stalled.sum() < R - 50
    lo, hi = np.max(L[~stalled]), np.min(L[stalled])
    assert lo < hi
    # the boundary lies within the gap the samples leave, up to the chi_D
    # series' distance from the exact mean
    assert lo * (1 - 1e-3) <= thr <= hi * (1 + 1e-3), (lo, thr, hi)
