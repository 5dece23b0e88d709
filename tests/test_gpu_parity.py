"""GPU path against the oracle, through the C-ABI (marked gpu).

Tolerances (derived in the design notes from the arithmetic):
  words, ranks, weights, member layout ........ bit-exact
  normals eps  |d| <= EPS_REL*|eps| + EPS_ABS  (exhaustive error of the
               hardware log2/sqrt/sin/cos over all 2^24 uniforms)
  fitness      |d| <= 1e-5 * S_j (S_j: sum of |terms|)
  one tell     max |dm| / max(|m|, lr) <= 1e-5, g within its error bound
"""
import math

import numpy as np
import pytest
import torch

from inputs import fitness_with_ties, random_state, to_oracle
from oracle import oracle as O

pytestmark = pytest.mark.gpu

EPS_REL, EPS_ABS = 3e-7, 8e-7


def _es():
    import paper_2212_04180_amd as P
    return P


def _cfg(**kw):
    P = _es()
    base = dict(num_dims=37, popsize=10, num_runs=1, sigma=0.1, lr=0.01, seed=5, init=P.INIT_UNIFORM,
                init_lo=-2.0, init_hi=2.0, problem=P.PROB_SPHERE)
    base.update(kw)
    return P.ESConfig(**base)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _assert_eps_close(got, ref, what=""):
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    bound = EPS_REL * np.abs(ref.astype(np.float64)) + EPS_ABS
    bad = np.nonzero(err > bound)[0]
    assert bad.size == 0, (what, bad[:5], got[bad[:5]], ref[bad[:5]])


# ---------------------------------------------------------------------------
# T0 / T1: the random stream
@pytest.mark.parametrize("D", [1, 3, 4, 13, 1000, 4099])
@pytest.mark.parametrize("seed,run,t,pair", [(0, 0, 0, 0), (7, 2, 5, 3), ((1 << 32) + 9, 1, 123456, 0)])
def test_noise_words_bit_exact_and_normals_close(D, seed, run, t, pair):
    P = _es()
    es = P.ES(_cfg(num_dims=D, popsize=8, num_runs=3, seed=seed))
    w, e = es.debug_noise(run, t, pair)
    w, e = _np(w).view(np.uint32), _np(e)
    nb = (D + 3) // 4
    ref_w = O.words(seed + run, O.DOM_NOISE, pair, t, 0, nb)
    np.testing.assert_array_equal(w, ref_w)
    ref_e = O.normals(seed + run, O.DOM_NOISE, pair, t, 0, D)
    _assert_eps_close(e, ref_e, (D, seed, run, t, pair))


def test_normals_error_statistics_large():
    # 2^22 normals: the error bound holds everywhere, and the errors are
    # unbiased (hardware and libm agree to within rounding on average).
    P = _es()
    D = 1 << 22
    es = P.ES(_cfg(num_dims=D, popsize=2, seed=11, problem=P.PROB_NONE))
    _, e = es.debug_noise(0, 3, 0)
    e = _np(e)
    ref = O.normals(11, O.DOM_NOISE, 0, 3, 0, D)
    _assert_eps_close(e, ref, "large")
    d = e.astype(np.float64) - ref
    assert abs(d.mean()) < 1e-8 and np.mean(e == ref) > 0.2


# ---------------------------------------------------------------------------
# initial mean, problem data, materialised ask
@pytest.mark.parametrize("lo,hi,R,D", [(-5.0, 5.0, 1, 16), (-2.0, 2.0, 1, 1000), (-5.12, 5.12, 7, 103)])
def test_init_uniform_bit_exact(lo, hi, R, D):
    P = _es()
    cfg = _cfg(num_dims=D, num_runs=R, init_lo=lo, init_hi=hi, seed=3)
    es = P.ES(cfg)
    m = _np(es.get_state()["m"])
    oc = to_oracle(cfg)
    for r in range(R):
        np.testing.assert_array_equal(m[r], O.init_mean(oc, r))


def test_init_zero_and_shift_vector():
    P = _es()
    cfg = _cfg(num_dims=1001, init=P.INIT_ZERO, problem=P.PROB_SHIFTED_SPHERE, seed=2)
    es = P.ES(cfg)
    st = es.get_state()
    assert np.all(_np(st["m"]) == 0) and np.all(_np(st["m1"]) == 0) and np.all(_np(st["v"]) == 0)
    _assert_eps_close(_np(es.problem_data()), O.problem_data(to_oracle(cfg)), "shift")


@pytest.mark.parametrize("D,N,R", [(5, 4, 1), (64, 6, 2), (130, 12, 3)])
def test_ask_materialised_layout(D, N, R):
    P = _es()
    cfg = _cfg(num_dims=D, popsize=N, num_runs=R, sigma=0.3, seed=9)
    es = P.ES(cfg)
    x = _np(es.ask(materialize=True))
    m = _np(es.get_state()["m"])
    oc = to_oracle(cfg)
    for r in range(R):
        ref = O.population(oc, r, 0, m[r])
        # x = fmaf(+-sigma, eps, m): error sigma*|d eps| plus one rounding
        err = np.abs(x[r].astype(np.float64) - ref)
        eps_abs = np.abs((ref - m[r]) / 0.3)
        bound = 0.3 * (EPS_REL * eps_abs + EPS_ABS) + np.spacing(np.abs(ref).astype(np.float32))
        assert np.all(err <= bound)
    # antithetic layout is exact: member j and j+N/2 mirror around m
    cfg0 = _cfg(num_dims=D, popsize=N, num_runs=R, sigma=0.3, seed=9, init=P.INIT_ZERO)
    x0 = _np(P.ES(cfg0).ask(materialize=True))
    np.testing.assert_array_equal(x0[:, : N // 2], -x0[:, N // 2:])


# ---------------------------------------------------------------------------
# T2: fused sample + evaluate
def _scale_terms(problem, x, s=None, a=10.0):
    x = x.astype(np.float64)
    if problem == O.PROB_SPHERE:
        return np.sum(x * x, -1)
    if problem == O.PROB_SHIFTED_SPHERE:
        return np.sum((x - s) ** 2, -1)
    if problem == O.PROB_ROSENBROCK:
        return np.sum(100 * (x[..., 1:] - x[..., :-1] ** 2) ** 2 + (1 - x[..., :-1]) ** 2, -1)
    return a * x.shape[-1] + np.sum(np.abs(x * x - a * np.cos(2 * np.pi * x)), -1)


@pytest.mark.parametrize("prob", ["sphere", "shifted", "rosenbrock", "rastrigin"])
@pytest.mark.parametrize("D,N,R", [(1, 2, 1), (2, 4, 2), (7, 6, 1), (16, 32, 1), (1003, 10, 2), (4100, 514, 1)])
def test_eval_matches_oracle(prob, D, N, R):
    P = _es()
    pmap = {"sphere": P.PROB_SPHERE, "shifted": P.PROB_SHIFTED_SPHERE, "rosenbrock": P.PROB_ROSENBROCK,
            "rastrigin": P.PROB_RASTRIGIN}
    cfg = _cfg(num_dims=D, popsize=N, num_runs=R, problem=pmap[prob], sigma=0.2, seed=21,
               init=P.INIT_ZERO if prob == "shifted" else P.INIT_UNIFORM)
    es = P.ES(cfg)
    es.ask()
    f = _np(es.eval())
    oc = to_oracle(cfg)
    m = _np(es.get_state()["m"])
    pdata = O.problem_data(oc) if prob == "shifted" else None
    for r in range(R):
        ref = O.eval_members(oc, r, 0, m[r], pdata, np.arange(N))
        S = _scale_terms(cfg.problem, O.population(oc, r, 0, m[r]), pdata)
        err = np.abs(f[r].astype(np.float64) - ref)
        assert np.all(err <= 1e-5 * S + 1e-30), (prob, D, N, r, err.max(), (err / np.maximum(S, 1e-30)).max())


# ---------------------------------------------------------------------------
# T0: ranks and weights from the same fp32 fitness
@pytest.mark.parametrize("N,R,maximize", [(2, 1, 0), (8, 3, 0), (64, 5, 1), (1024, 2, 0), (2048, 1, 1), (16384, 1, 0)])
def test_ranks_and_weights_bit_exact(N, R, maximize):
    P = _es()
    cfg = _cfg(num_dims=9, popsize=N, num_runs=R, maximize=maximize, problem=P.PROB_NONE)
    es = P.ES(cfg)
    f = fitness_with_ties(N + R, R, N, ties=True, specials=True)
    es.ask()
    es.tell(torch.tensor(f, device="cuda"))
    y, rk = es.shaped()
    y, rk = _np(y), _np(rk)
    for r in range(R):
        np.testing.assert_array_equal(rk[r], O.ranks(f[r], maximize))
        np.testing.assert_array_equal(y[r], O.shape(f[r], maximize))


# ---------------------------------------------------------------------------
# T3: one tell from the same state and the same fitness
@pytest.mark.parametrize("D,N,R,t", [(6, 4, 1, 0), (37, 10, 2, 5), (1000, 256, 1, 17), (4099, 2048, 1, 2)])
def test_tell_matches_oracle(D, N, R, t):
    P = _es()
    cfg = _cfg(num_dims=D, popsize=N, num_runs=R, problem=P.PROB_NONE, sigma=0.05, lr=0.005,
               flags=P.FLAG_KEEP_GRAD, seed=77)
    es = P.ES(cfg)
    m, m1, v, _ = random_state(D + N, R, D, t)
    es.set_state(*(torch.tensor(a, device="cuda") for a in (m, m1, v)), t)
    f = fitness_with_ties(D * N, R, N, ties=False)
    es.ask()
    es.tell(torch.tensor(f, device="cuda"))
    g = _np(es.grad())
    st = es.get_state()
    assert st["t"] == t + 1
    mg, m1g, vg = _np(st["m"]), _np(st["m1"]), _np(st["v"])
    oc = to_oracle(cfg)
    for r in range(R):
        y = O.shape(f[r])
        gref = O.grad(oc, r, t, y)
        # bound: noise error propagated through the weighted sum + fp32 sums
        w = (y[: N // 2].astype(np.float64) - y[N // 2:])
        E = np.stack([O.noise(oc, r, t, p) for p in range(N // 2)]).astype(np.float64)
        ns = N * np.float64(np.float32(0.05))
        bound = (np.abs(w) @ (EPS_REL * np.abs(E) + EPS_ABS) + 1e-6 * (np.abs(w) @ np.abs(E))) / ns
        assert np.all(np.abs(g[r] - gref) <= bound + 1e-12), (r, np.max(np.abs(g[r] - gref) - bound))
        mr, m1r, vr = O.adam(oc, t, gref, m[r], m1[r], v[r])
        den = np.maximum(np.abs(mr), cfg.lr)
        assert np.max(np.abs(mg[r] - mr) / den) <= 1e-5
        assert np.all(np.abs(m1g[r] - m1r) <= 0.1 * bound + 2 * np.spacing(np.abs(m1r)))
        # Adam itself is bit-exact given the same g
        ma, m1a, va = O.adam(oc, t, g[r], m[r], m1[r], v[r])
        np.testing.assert_array_equal(mg[r], ma)
        np.testing.assert_array_equal(m1g[r], m1a)
        np.testing.assert_array_equal(vg[r], va)


def test_split_tell_repeated_and_deterministic():
    """A geometry with few groups of Philox blocks (D = 4099, N = 2048, two
    runs), whose pairs the gradient kernel spreads over several workgroups per
    block group: three consecutive tells, each checked against the oracle from
    the state the GPU reached, and bit-identical across two handles (the
    workgroups' partial sums meet in a fixed order whichever arrives last)."""
    P = _es()
    D, N, R = 4099, 2048, 2
    cfg = _cfg(num_dims=D, popsize=N, num_runs=R, problem=P.PROB_NONE, sigma=0.05, lr=0.005,
               flags=P.FLAG_KEEP_GRAD, seed=5)
    a, b = P.ES(cfg), P.ES(cfg)
    oc = to_oracle(cfg)
    for t in range(3):
        f = fitness_with_ties(100 + t, R, N, ties=False)
        st0 = a.get_state()
        m0, m10, v0 = _np(st0["m"]), _np(st0["m1"]), _np(st0["v"])
        for es in (a, b):
            es.ask()
            es.tell(torch.tensor(f, device="cuda"))
        ga, gb = _np(a.grad()), _np(b.grad())
        np.testing.assert_array_equal(ga, gb)
        sa, sb = a.get_state(), b.get_state()
        for k in ("m", "m1", "v"):
            np.testing.assert_array_equal(_np(sa[k]), _np(sb[k]))
        mg = _np(sa["m"])
        for r in range(R):
            y = O.shape(f[r])
            gref = O.grad(oc, r, t, y)
            assert np.max(np.abs(ga[r] - gref)) <= 1e-4 * np.max(np.abs(gref)), (t, r)
            mr, _, _ = O.adam(oc, t, gref, m0[r], m10[r], v0[r])
            assert np.max(np.abs(mg[r] - mr) / np.maximum(np.abs(mr), cfg.lr)) <= 1e-5, (t, r)
            ma, _, _ = O.adam(oc, t, ga[r], m0[r], m10[r], v0[r])
            np.testing.assert_array_equal(mg[r], ma)
