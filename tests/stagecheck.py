"""Stage-by-stage comparison of one library handle with the oracle (GPU tests).

Each generation the oracle takes the GPU's state (mean, moments or paths,
per-dimension sigma, velocity, run sigma and lr); both sides evaluate the same
population; the oracle's tell takes the GPU's fitness vector, so both rank the
same values; then every updated quantity is compared.  The bars follow from
the normals' error bound (T1: |dz| <= 3e-7 |z| + 8e-7, |z| <= 5.77, so
|dz| <= DZ = 2.6e-6) propagated through each step, plus fp32 rounding:

  fitness      |df| <= 1e-5 S + DZ sum_d s_d |df/dx_d| (+ second order)
  shaping      bit-exact (centered, raw, rank tables), z-score within 1 ulp
  g (OpenAI-ES, PGPE; kept with ES_FLAG_KEEP_GRAD)
               within sum_p |a_p| (3e-7 |z| + 8e-7) scaled as g, + 1e-6 rel.
  Adam         bit-exact given the kernel's g
  ClipUp       velocity within 1e-5 of max(speed, |v|); m = m - v exactly
  PGPE sigma   1e-5 rel + sigma_lr sigma_d (sum_p |b_p| 2 |z| DZ) / P
  SNES         m: 1e-5 rel (floor lr/10) + lr sigma_d sum_p |a_p| DZ;
               sigma: 1e-5 rel + (sigma_lr/2) sum_p |b_p| 2 |z| DZ
  Sep-CMA-ES   m: 1e-5 rel (floor 1e-3) + s_d DZ (weights sum to 1);
               p_sigma, p_c: a_s DZ, a_c DZ + 2 ulp; C: 1e-5 rel +
               C (c_mu 2 |z| DZ + c1 2 |p_c| a_c DZ); sigma 1e-5 rel.
"""
import math

import numpy as np
import torch

from inputs import to_oracle
from oracle import oracle as O

EPS_REL, EPS_ABS = 3e-7, 8e-7
DZ = EPS_REL * 5.77 + EPS_ABS
ZMAX = 5.77


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _ulps(a, b):
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    return np.abs(a.astype(np.float64) - b.astype(np.float64)) / np.spacing(np.maximum(np.abs(a), np.abs(b)))


def _terms_and_slopes(problem, x, s, a):
    """Sum of |terms| and sum_d |df/dx_d| s_d-weighted later; x: [N][D]."""
    if problem == O.PROB_SPHERE:
        return np.sum(x * x, -1), 2.0 * np.abs(x), 2.0 * np.ones_like(x)
    if problem == O.PROB_SHIFTED_SPHERE:
        d = x - s
        return np.sum(d * d, -1), 2.0 * np.abs(d), 2.0 * np.ones_like(x)
    if problem == O.PROB_ROSENBROCK:
        u = x[:, 1:] - x[:, :-1] ** 2
        terms = 100.0 * u * u + (1.0 - x[:, :-1]) ** 2
        g = np.zeros_like(x)
        g[:, :-1] += 400.0 * np.abs(x[:, :-1] * u) + 2.0 * np.abs(1.0 - x[:, :-1])
        g[:, 1:] += 200.0 * np.abs(u)
        h = np.zeros_like(x)
        h[:, :-1] += 1200.0 * x[:, :-1] ** 2 + 400.0 * np.abs(x[:, 1:]) + 202.0
        h[:, 1:] += 200.0
        return np.sum(np.abs(terms), -1), g, h
    terms = a + np.abs(x * x) + a * np.abs(np.cos(2 * np.pi * x))
    return np.sum(terms, -1), 2.0 * np.abs(x) + 2 * np.pi * a, 2.0 + 4 * np.pi ** 2 * a * np.ones_like(x)


def _fitness_bound(cfg, x, scale, pdata):
    x = x.astype(np.float64)
    s = pdata.astype(np.float64) if pdata is not None else None
    S, g, h = _terms_and_slopes(cfg.problem, x, s, float(cfg.rastrigin_a))
    dx = DZ * np.broadcast_to(np.asarray(scale, np.float64), x.shape)
    return 1e-5 * S + np.sum(g * dx, -1) + 0.5 * np.sum(h * dx * dx, -1) + 1e-30


def grad_bound(oc, r, t, y):
    """Per-dimension bound on |g_gpu - g_oracle| for OpenAI-ES: the normals'
    error (T1) summed over the pairs' folded weights, plus fp32 rounding of
    the kernel's sums (1e-6 of the same sum)."""
    N = oc.popsize
    w = y[: N // 2].astype(np.float64) - y[N // 2:]
    S = O.abs_noise_sum(oc, r, t, w.astype(np.float32))
    return ((EPS_REL + 1e-6) * S + EPS_ABS * np.sum(np.abs(w))) / (N * np.float64(np.float32(oc.sigma)))


def adam_tolerance(oc, t, g, m1, v, delta):
    """Per-dimension bound on the Adam step's difference when g is known to
    within delta: lr |dq| <= lr delta sup |q'(g')| over |g' - g| <= delta, with
    q = mhat / (sqrt(vhat) + eps), mhat = a + b g', vhat = c + d g'^2 and
    |q'| <= |b| / S + (|a| + |b| g') d g' / S^3, S = sqrt(vhat) (an upper bound:
    eps only enlarges the denominator).  Where g may be 0 at t = 0 (c = 0)
    the bound is infinite: the step there follows the sign of g, a near-tie.
    Adam's step is scale-free in g, so this term, not the fp32 rounding, sets
    the tolerance wherever |g| is small."""
    b1, b2 = np.float64(np.float32(oc.beta1)), np.float64(np.float32(oc.beta2))
    tp = t + 1
    bc1, bc2 = np.float64(np.float32(1 - b1 ** tp)), np.float64(np.float32(1 - b2 ** tp))
    a = b1 * m1.astype(np.float64) / bc1
    b = (1 - b1) / bc1
    c = b2 * v.astype(np.float64) / bc2
    d = (1 - b2) / bc2
    g = np.abs(g.astype(np.float64))
    gmin = np.maximum(g - delta, 0.0)
    gmax = g + delta
    S = np.sqrt(c + d * gmin * gmin)
    with np.errstate(divide="ignore", invalid="ignore"):
        dq = np.where(S > 0, abs(b) / S + (np.abs(a) + abs(b) * gmax) * d * gmax / S ** 3, np.inf)
    return np.float64(np.float32(oc.lr)) * delta * dq


def _noise_rows(oc, r, t, rows, D):
    return np.stack([O.normals(oc.seed + r, O.DOM_NOISE, int(p), t, 0, D) for p in rows]).astype(np.float64)


def run(P, cfg, T):
    """T generations of cfg on the GPU and in the oracle, compared after each."""
    strategy, optimizer = cfg.strategy, cfg.optimizer
    clip = optimizer == P.OPT_CLIPUP and strategy != P.STRAT_SNES
    adam = optimizer == P.OPT_ADAM and strategy in (P.STRAT_OPENAI_ES, P.STRAT_PGPE)
    keep = bool(cfg.flags & P.FLAG_KEEP_GRAD)
    es = P.ES(cfg)
    oc = to_oracle(cfg)
    ref = O.OracleES(oc)
    D, N, R = cfg.num_dims, cfg.popsize, cfg.num_runs
    Pp = N // 2
    pdata = O.problem_data(oc) if cfg.problem == P.PROB_SHIFTED_SPHERE else None
    for t in range(T):
        st = es.get_state()
        m0, m10, v0 = _np(st["m"]), _np(st["m1"]), _np(st["v"])
        sig = vel = None
        if strategy != P.STRAT_OPENAI_ES or clip:
            sg, ve = es.strategy_state(sigma=strategy != P.STRAT_OPENAI_ES, velocity=clip)
            sig = _np(sg) if sg is not None else None
            vel = _np(ve) if ve is not None else None
        ref.set_state(m0, m10, v0, st["t"], sig=sig, vel=vel)
        ref.set_hparams(*es.get_hparams())
        rcfg = [ref.run_cfg(r) for r in range(R)]
        scales = [ref.scale(r) if strategy != P.STRAT_OPENAI_ES else np.float32(ref.sigma[r]) for r in range(R)]
        es.ask()
        f = _np(es.eval())
        fr = ref.eval()
        xs = ref.ask()
        for r in range(R):
            bound = _fitness_bound(cfg, xs[r], scales[r], pdata)
            err = np.abs(f[r].astype(np.float64) - fr[r])
            assert np.all(err <= bound), (t, r, "fitness", float(np.max(err / bound)))
        es.tell(torch.tensor(f, device="cuda"))
        y = _np(es.shaped()[0])
        ref.tell(f)
        st = es.get_state()
        m, m1, v = _np(st["m"]), _np(st["m1"]), _np(st["v"])
        g = _np(es.grad()) if keep else None
        for r in range(R):
            # shaping from the same fitness
            rk = O.ranks(f[r], cfg.maximize)
            if strategy == P.STRAT_SNES:
                yr = O.snes_table(N, cfg.snes_temperature)[N - 1 - rk]
                np.testing.assert_array_equal(y[r], yr)
            elif strategy == P.STRAT_SEP_CMA:
                w = O.cma_weights(oc).astype(np.float32)
                np.testing.assert_array_equal(y[r], np.where(rk < len(w), w[np.minimum(rk, len(w) - 1)], 0))
            else:
                yr = O.shape_full(f[r], None, cfg.maximize, cfg.shaping)
                if cfg.shaping == P.SHAPE_Z_SCORE:
                    assert np.all(_ulps(y[r], yr) <= 1.0), (t, r, "z-score")
                else:
                    np.testing.assert_array_equal(y[r], yr)
            a_p = (y[r][:Pp].astype(np.float64) - y[r][Pp:]) if strategy != P.STRAT_SEP_CMA else None
            b_p = (y[r][:Pp].astype(np.float64) + y[r][Pp:]) if strategy in (P.STRAT_PGPE, P.STRAT_SNES) else None
            if strategy == P.STRAT_PGPE:
                b_p = b_p / 2.0 - np.mean(y[r].astype(np.float64))
            E = _noise_rows(oc, r, t, range(Pp), D) if strategy != P.STRAT_SEP_CMA else None
            if strategy in (P.STRAT_OPENAI_ES, P.STRAT_PGPE):
                # g against the oracle's estimate from the same weights
                aw = np.abs(a_p) @ (EPS_REL * np.abs(E) + EPS_ABS) + 1e-6 * (np.abs(a_p) @ np.abs(E))
                if strategy == P.STRAT_OPENAI_ES:
                    gref = O.grad(rcfg[r], r, t, y[r]).astype(np.float64)
                    gb = aw / (N * float(rcfg[r].sigma))
                else:
                    A, _ = O.noise_sums(rcfg[r], r, t, a_p.astype(np.float32), b_p.astype(np.float32))
                    sd = sig[r].astype(np.float64)
                    gref = sd * A / N
                    gb = sd * aw / N
                if keep:
                    assert np.all(np.abs(g[r] - gref) <= gb + 2 * np.spacing(np.abs(gref))), (t, r, "g")
                    if adam:
                        ma, m1a, va = O.adam(rcfg[r], t, g[r], m0[r], m10[r], v0[r])
                        np.testing.assert_array_equal(m[r], ma)
                        np.testing.assert_array_equal(m1[r], m1a)
                        np.testing.assert_array_equal(v[r], va)
                elif adam:
                    # without the kernel's g: the tell tier on the mean
                    den = np.maximum(np.abs(ref.m[r]), rcfg[r].lr)
                    assert np.max(np.abs(m[r] - ref.m[r]) / den) <= 1e-5, (t, r, "m")
                if strategy == P.STRAT_PGPE:
                    sref = ref.sig[r].astype(np.float64)
                    bb = np.abs(b_p) @ (2 * ZMAX * DZ * np.ones_like(E))
                    tol = 1e-5 * sref + cfg.sigma_lr * sig[r] * bb / Pp
                    assert np.all(np.abs(_np(es.strategy_state()[0])[r] - sref) <= tol), (t, r, "pgpe sigma")
            if clip:
                ve = _np(es.strategy_state(sigma=False, velocity=True)[1])[r]
                bound = 1e-5 * max(cfg.clipup_max_speed, float(np.max(np.abs(ref.vel[r]))))
                assert np.max(np.abs(ve - ref.vel[r])) <= bound, (t, r, "velocity")
                np.testing.assert_array_equal(m[r], (m0[r] - ve).astype(np.float32))
            if strategy == P.STRAT_SNES:
                sd = sig[r].astype(np.float64)
                tol = 1e-5 * np.maximum(np.abs(ref.m[r]), rcfg[r].lr * 0.1) + rcfg[r].lr * sd * np.sum(np.abs(a_p)) * DZ
                assert np.all(np.abs(m[r] - ref.m[r]) <= tol), (t, r, "snes m")
                sref = ref.sig[r].astype(np.float64)
                tol = sref * (1e-5 + cfg.sigma_lr / 2 * np.sum(np.abs(b_p)) * 2 * ZMAX * DZ)
                assert np.all(np.abs(_np(es.strategy_state()[0])[r] - sref) <= tol), (t, r, "snes sigma")
            if strategy == P.STRAT_SEP_CMA:
                w = O.cma_weights(oc)
                mu_eff = 1.0 / np.sum(w ** 2)
                c_s = (mu_eff + 2.0) / (D + mu_eff + 5.0)
                a_s = math.sqrt(c_s * (2.0 - c_s) * mu_eff)
                c_c = (4.0 + mu_eff / D) / (D + 4.0 + 2.0 * mu_eff / D)
                a_c = math.sqrt(c_c * (2.0 - c_c) * mu_eff)
                sd = np.asarray(scales[r], np.float64)
                tol = 1e-5 * np.maximum(np.abs(ref.m[r]), 1e-3) + sd * DZ
                assert np.all(np.abs(m[r] - ref.m[r]) <= tol), (t, r, "cma m")
                assert np.all(np.abs(m1[r] - ref.m1[r]) <= a_s * DZ + 2 * np.spacing(np.abs(ref.m1[r]))), (t, r, "p_s")
                assert np.all(np.abs(v[r] - ref.v[r]) <= 1e-5 * np.abs(ref.v[r]) + a_c * DZ
                              + 2 * np.spacing(np.abs(ref.v[r]))), (t, r, "p_c")
                C = _np(es.strategy_state()[0])[r]
                Cr = ref.sig[r].astype(np.float64)
                tol = 1e-5 * Cr + sig[r] * (2 * ZMAX * DZ + 2 * np.abs(ref.v[r]) * a_c * DZ)
                assert np.all(np.abs(C - Cr) <= tol), (t, r, "C")
        sg, lr = es.get_hparams()
        assert np.all(np.abs(sg - ref.sigma) <= 1e-5 * ref.sigma), (t, "sigma")
        np.testing.assert_array_equal(lr, ref.lr)
    return es, ref
