"""Pins of the oracle's tell step: the FD gradient estimator of Sec. 2.1 against
closed forms and its expectation, and the Adam update against torch.optim.Adam
and the textbook formula (CPU only)."""
import math

import numpy as np
import pytest
import torch
from scipy import integrate, stats

from oracle import oracle as O


def _tell_with(cfg, fit_fn, t=0, m=None):
    es = O.OracleES(cfg)
    if m is not None:
        es.set_state(m[None, :], np.zeros_like(m)[None, :], np.zeros_like(m)[None, :], t)
    x = es.ask()[0].astype(np.float64)
    f = np.array([fit_fn(xj) for xj in x], np.float32)
    m0 = es.m[0].copy()
    out = es.tell(f[None, :])
    return x, f, out["g"][0], m0, es


def test_grad_linear_raw_converges_to_a():
    # f = a.x, raw shaping: g = (2/N) sum_p (a.eps_p) eps_p, E[g] = a,
    # sd_i = sqrt((|a|^2 + a_i^2) / (N/2)).
    D, N = 8, 20000
    a = np.array([1.0, -2.0, 0.5, 0.0, 3.0, -0.25, 1.5, -1.0])
    cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.05, init=O.INIT_ZERO, problem=O.PROB_NONE,
                         shaping=O.SHAPE_RAW, seed=123)
    _, _, g, _, _ = _tell_with(cfg, lambda x: float(a @ x))
    sd = np.sqrt((a @ a + a * a) / (N / 2))
    assert np.all(np.abs(g - a) <= 5 * sd), (g, a, sd)


def test_grad_sphere_raw_exact_identity_and_mean():
    # Sphere, raw shaping: f(m+s e) - f(m-s e) = 4 s m.e exactly, so
    # g = (4/N) sum_p (m.eps_p) eps_p per sample; its mean is 2m.
    D, N = 6, 2000
    cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=0.1, init=O.INIT_UNIFORM, init_lo=-5, init_hi=5,
                         problem=O.PROB_SPHERE, shaping=O.SHAPE_RAW, seed=5)
    es = O.OracleES(cfg)
    m = es.m[0].astype(np.float64)
    out = es.tell(None)
    g = out["g"][0].astype(np.float64)
    eps = np.stack([O.noise(cfg, 0, 0, p) for p in range(N // 2)]).astype(np.float64)
    ident = (4.0 / N) * ((eps @ m)[:, None] * eps).sum(0)
    # fp32 rounding of x and f: |dg| <~ (N/2) * 2 ulp(f) / (N sigma) per unit |eps|
    fmax = float(np.max(out["fitness"]))
    tol = 3 * np.spacing(np.float32(fmax)) / cfg.sigma * np.abs(eps).mean(0) * 2
    assert np.all(np.abs(g - ident) <= tol + 1e-6), (g, ident, tol)
    sd = np.sqrt(4 * (m @ m + m * m) / (N / 2))
    assert np.all(np.abs(g - 2 * m) <= 5 * sd)


def test_grad_centered_rank_linear_expectation():
    # Centered ranks on f = a.x: with u = a.eps/|a| the ranks only see the
    # symmetric set {+-u_p}; summing (rank/(N-1) - 1/2) z over it gives
    # E[a_hat . g] * sigma = (M sqrt(2/pi) + M(M-1) E[max(|u1|,|u2|)]) / (N (N-1)),
    # M = N/2, with E[max] = integral of 1 - (2 Phi(t) - 1)^2 (computed here).
    emax = integrate.quad(lambda t: 1 - (2 * stats.norm.cdf(t) - 1) ** 2, 0, 40)[0]
    D, N, sigma, S = 5, 32, 0.3, 400
    M = N // 2
    cN = (M * math.sqrt(2 / math.pi) + M * (M - 1) * emax) / (N * (N - 1))
    assert cN == pytest.approx(((N - 2) / (2 * math.sqrt(math.pi)) + 1 / math.sqrt(2 * math.pi)) / (N - 1), rel=1e-9)
    a = np.array([2.0, -1.0, 0.5, 0.0, 1.0])
    ah = a / np.linalg.norm(a)
    proj, orth = [], []
    for s in range(S):
        cfg = O.OracleConfig(num_dims=D, popsize=N, sigma=sigma, init=O.INIT_ZERO, problem=O.PROB_NONE, seed=1000 + s)
        _, _, g, _, _ = _tell_with(cfg, lambda x: float(a @ x))
        g = g.astype(np.float64)
        proj.append(ah @ g * sigma)
        orth.append(g[3] * sigma)  # a_3 = 0 and e_3 is orthogonal to a
    proj, orth = np.array(proj), np.array(orth)
    assert abs(proj.mean() - cN) < 5 * proj.std() / math.sqrt(S)
    assert abs(orth.mean()) < 5 * orth.std() / math.sqrt(S)


def test_minimisation_moves_mean_downhill():
    # Listing 1: minimisation by default -- the mean moves against the gradient.
    cfg = O.OracleConfig(num_dims=4, popsize=64, sigma=0.1, lr=0.05, init=O.INIT_ZERO, problem=O.PROB_NONE, seed=3)
    a = np.array([1.0, -1.0, 2.0, 0.0])
    x, f, g, m0, es = _tell_with(cfg, lambda x: float(a @ x))
    step = es.m[0] - m0
    assert step @ a < 0
    cfgM = O.OracleConfig(num_dims=4, popsize=64, sigma=0.1, lr=0.05, init=O.INIT_ZERO, problem=O.PROB_NONE,
                          seed=3, maximize=1)
    x, f, g, m0, es = _tell_with(cfgM, lambda x: float(a @ x))
    assert (es.m[0] - m0) @ a > 0


def test_adam_first_step_is_signed_lr():
    cfg = O.OracleConfig(num_dims=5, popsize=2, lr=0.01)
    g = np.array([0.3, -2.0, 1e-3, -7.5, 100.0], np.float32)
    m = np.array([1.0, 2.0, 3.0, -4.0, 0.0], np.float32)
    m2, m1, v = O.adam(cfg, 0, g, m, np.zeros(5, np.float32), np.zeros(5, np.float32))
    want = m - 0.01 * g / (np.abs(g) + 1e-8)
    assert np.all(np.abs(m2 - want) <= 2e-7 * np.maximum(1, np.abs(m))), (m2, want)
    # (1 - beta) is taken of the fp32 betas
    np.testing.assert_allclose(m1, (1 - float(np.float32(0.9))) * g.astype(np.float64), rtol=1e-6)
    np.testing.assert_allclose(v, (1 - float(np.float32(0.999))) * g.astype(np.float64) ** 2, rtol=1e-6)


def test_adam_matches_torch_and_textbook():
    rng = np.random.default_rng(7)
    n, T = 64, 30
    lr, b1, b2, eps = 0.005, 0.9, 0.999, 1e-8
    cfg = O.OracleConfig(num_dims=n, popsize=2, lr=lr, beta1=b1, beta2=b2, eps=eps)
    m = rng.normal(size=n).astype(np.float32)
    m1 = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    p = torch.tensor(m.copy(), dtype=torch.float32, requires_grad=True)
    opt = torch.optim.Adam([p], lr=lr, betas=(b1, b2), eps=eps, foreach=False)
    mt, m1t, vt = m.astype(np.float64), np.zeros(n), np.zeros(n)
    b1f, b2f = float(np.float32(b1)), float(np.float32(b2))
    for t in range(T):
        g = (rng.normal(size=n) * 10 ** rng.uniform(-3, 1, size=n)).astype(np.float32)
        m, m1, v = O.adam(cfg, t, g, m, m1, v)
        p.grad = torch.tensor(g)
        opt.step()
        gd = g.astype(np.float64)
        m1t = b1f * m1t + (1 - b1f) * gd
        vt = b2f * vt + (1 - b2f) * gd * gd
        mt = mt - lr * (m1t / (1 - b1f ** (t + 1))) / (np.sqrt(vt / (1 - b2f ** (t + 1))) + eps)
        np.testing.assert_allclose(m, p.detach().numpy(), rtol=0, atol=4e-7 * max(1.0, float(np.abs(m).max())))
        np.testing.assert_allclose(m, mt, rtol=0, atol=1e-6 * max(1.0, float(np.abs(mt).max())))
