"""Neuroevolution fitness on the GPU (bf16 matrix cores) against the oracle's
bf16-emulating CPU forward, and the gradient / Adam / ClipUp tell of the
neuroevolution workload (marked gpu).

Fitness bars.  The contract tier is |df| <= 2e-2 |f| (f = -MSE, a sum of
non-negative terms): the two sides differ by the normals' error (which can
flip a weight's bf16 rounding), the fp32-vs-fp64 accumulation, the hardware
exp/rcp tanh against libm, and the bf16 rounding decisions those flip.  With
the weights taken from the GPU's own materialised population (es_ask), both
sides round the same fp32 weights, and what is left is bounded far tighter:
  - fp32 accumulation of K <= 256 products, relative error <= K 2^-24 of the
    sum of |terms| per dot product, propagated through two tanh layers
    (|tanh'| <= 1): about 3e-5 of the output scale;
  - the hardware tanh (exp2 and rcp, each within 1 ulp) is within 4e-7 of
    libm's, so a bf16-rounded activation differs by one bf16 ulp (2^-8
    relative) only where the exact value lies within 4e-7 of a rounding
    boundary; each such flip moves the outputs by at most 2^-8 |h| |W|;
  - with about 1e-3 of the 131,072 activations of a member flipped and their
    signs random, the MSE moves by well under 1e-4 of itself.
That bar (TIGHT = 1e-3, ten times the estimate) fails for a wrong scale of a
single layer's output by 1% or more (the MSE then moves by ~2% of itself).
The observed maxima are printed beside each bar.
"""
import numpy as np
import pytest
import torch

import stagecheck
from inputs import to_oracle
from oracle import oracle as O

pytestmark = pytest.mark.gpu

TOL = 2e-2
TIGHT = 1e-3
EPS_REL, EPS_ABS = 3e-7, 8e-7
# first flat index of b1, W2, b2, W3, b3 in the 64-256-256-16 layout
MLP_BOUNDS = [16384, 16640, 82176, 82432, 86528]


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _cfg(**kw):
    import paper_2212_04180_amd as P
    base = dict(num_dims=86544, popsize=8, num_runs=1, sigma=0.02, lr=0.01, seed=3, init=P.INIT_FANIN_NORMAL,
                problem=P.PROB_MLP, maximize=1, mlp_batch=256, mlp_bf16=1)
    base.update(kw)
    return P.ESConfig(**base)


def test_teacher_and_init_match_oracle():
    import paper_2212_04180_amd as P
    cfg = _cfg()
    es = P.ES(cfg)
    oc = to_oracle(cfg)
    teacher = _np(es.problem_data())
    ref = O.problem_data(oc)
    err = np.abs(teacher.astype(np.float64) - ref)
    assert np.all(err <= 3e-7 * np.abs(ref) + 1e-7)  # normal error bound x (1/8 or 1/16)
    m = _np(es.get_state()["m"])[0]
    mr = O.init_mean(oc, 0)
    assert np.all(np.abs(m.astype(np.float64) - mr) <= 3e-7 * np.abs(mr) + 1e-7)
    assert np.all(m[16384:16640] == 0) and np.all(m[86528:] == 0)  # biases


@pytest.mark.parametrize("N,R,t", [(8, 1, 0), (6, 2, 3)])
def test_fitness_all_members(N, R, t):
    import paper_2212_04180_amd as P
    cfg = _cfg(popsize=N, num_runs=R)
    es = P.ES(cfg)
    oc = to_oracle(cfg)
    if t:
        es.set_state(*(s for s in (es.get_state()[k] for k in ("m", "m1", "v"))), t)
    es.ask()
    f = _np(es.eval())
    m = _np(es.get_state()["m"])
    teacher = O.problem_data(oc)
    for r in range(R):
        ref = O.eval_members(oc, r, t, m[r], teacher, np.arange(N))
        assert np.all(f[r] < 0)
        rel = np.abs(f[r] - ref) / np.abs(ref)
        print(f"run {r}: max relative fitness error {rel.max():.3e} (bar {TOL})", flush=True)
        assert np.all(rel <= TOL), (r, rel)


@pytest.mark.parametrize("N,t", [(8, 0), (10, 5)])
def test_fitness_same_weights_tight(N, t):
    """The oracle's forward on the GPU's materialised members (the same fp32
    weights on both sides) within the tight bar."""
    import paper_2212_04180_amd as P
    cfg = _cfg(popsize=N)
    es = P.ES(cfg)
    oc = to_oracle(cfg)
    if t:
        st = es.get_state()
        es.set_state(st["m"], st["m1"], st["v"], t)
    x = _np(es.ask(materialize=True))[0]
    f = _np(es.eval())[0]
    YT = O.mlp_teacher_out(oc, O.problem_data(oc), t)
    ref = np.array([O.mlp_fitness(oc, x[j], t, YT) for j in range(N)])
    rel = np.abs(f - ref) / np.abs(ref)
    print(f"same weights: max relative fitness error {rel.max():.3e} (bar {TIGHT})", flush=True)
    assert np.all(rel <= TIGHT), rel


def test_fitness_sampled_members_full_population():
    """The neuroevolution workload at full size (N = 1024): sampled members,
    both signs of a pair."""
    import paper_2212_04180_amd as P
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get("mlp_teacher")
    es = P.ES(cfg)
    oc = to_oracle(cfg)
    es.run(2)  # move off the initial mean
    es.ask()
    f = _np(es.eval())[0]
    st = es.get_state()
    m = _np(st["m"])[0]
    js = np.array([0, 1, 511, 512, 513, 1023])
    ref = O.eval_members(oc, 0, st["t"], m, O.problem_data(oc), js)
    rel = np.abs(f[js] - ref) / np.abs(ref)
    print(f"N=1024 sampled: max relative fitness error {rel.max():.3e} (bar {TOL})", flush=True)
    assert np.all(rel <= TOL), rel
    assert np.all(np.isfinite(f)) and np.all(f < 0)


def _mlp_windows(D):
    out = [(0, 64)]
    for b in MLP_BOUNDS:
        out.append((b - 32, min(64, D - (b - 32))))
    out.append((D - 40, 40))
    return out


@pytest.mark.parametrize("optimizer", ["adam", "clipup"])
def test_mlp_tell_matches_oracle(optimizer):
    """The neuroevolution workload's tell (D = 86,544, N = 1024) against the
    oracle, after a first generation so that the gradient launch carries the
    next generation's teacher rows in front of its gradient workgroups and is
    split and folded: g on windows straddling every layer boundary and the
    tail within its propagated bound (the normals' error summed over the
    pairs' weights, plus fp32 rounding), shaped weights bit-exact, the Adam
    step bit-exact given the kernel's g and within the tell tier given the
    oracle's; ClipUp: the velocity rule over the whole vector and m - v."""
    import dataclasses

    import paper_2212_04180_amd as P
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get("mlp_teacher")
    kw = dict(flags=P.FLAG_KEEP_GRAD)
    if optimizer == "clipup":
        kw.update(optimizer=P.OPT_CLIPUP, clipup_max_speed=0.05, clipup_momentum=0.9)
    cfg = dataclasses.replace(cfg, **kw)
    es = P.ES(cfg)
    oc = to_oracle(cfg)
    D, N = cfg.num_dims, cfg.popsize
    es.step()
    worst = 0.0
    for t in (1, 2):
        st = es.get_state()
        assert st["t"] == t
        m0, m10, v0 = _np(st["m"])[0], _np(st["m1"])[0], _np(st["v"])[0]
        vel0 = _np(es.strategy_state(sigma=False, velocity=True)[1])[0].astype(np.float64) if optimizer == "clipup" else None
        es.ask()
        f = _np(es.eval())
        es.tell(torch.tensor(f, device="cuda"))
        y = _np(es.shaped()[0])[0]
        np.testing.assert_array_equal(y, O.shape(f[0], maximize=1))
        g = _np(es.grad())[0]
        st = es.get_state()
        mg, m1g, vg = _np(st["m"])[0], _np(st["m1"])[0], _np(st["v"])[0]
        w = y[: N // 2].astype(np.float64) - y[N // 2:]
        ns = N * np.float64(np.float32(cfg.sigma))
        for d0, nd in _mlp_windows(D):
            sl = slice(d0, d0 + nd)
            gref = O.grad(oc, 0, t, y, d0, nd).astype(np.float64)
            E = np.stack([O.noise(oc, 0, t, p, d0, nd) for p in range(N // 2)]).astype(np.float64)
            bound = (np.abs(w) @ (EPS_REL * np.abs(E) + EPS_ABS) + 1e-6 * (np.abs(w) @ np.abs(E))) / ns
            err = np.abs(g[sl] - gref)
            worst = max(worst, float(np.max(err / (bound + 1e-12))))
            assert np.all(err <= bound + 1e-12), (t, d0, float(np.max(err / bound)))
            if optimizer == "adam":
                mr, _, _ = O.adam(oc, t, gref.astype(np.float32), m0[sl], m10[sl], v0[sl])
                prop = stagecheck.adam_tolerance(oc, t, gref, m10[sl], v0[sl], bound)
                assert np.all(np.abs(mg[sl] - mr) <= 1e-5 * np.maximum(np.abs(mr), cfg.lr) + prop), (t, d0)
        if optimizer == "adam":
            ma, m1a, va = O.adam(oc, t, g, m0, m10, v0)
            np.testing.assert_array_equal(mg, ma)
            np.testing.assert_array_equal(m1g, m1a)
            np.testing.assert_array_equal(vg, va)
        else:
            vel = _np(es.strategy_state(sigma=False, velocity=True)[1])[0].astype(np.float64)
            gd = g.astype(np.float64)
            raw = cfg.clipup_momentum * vel0 + cfg.lr * gd / np.linalg.norm(gd)
            scale = min(1.0, cfg.clipup_max_speed / np.linalg.norm(raw))
            assert np.max(np.abs(vel - raw * scale)) <= 1e-5 * np.max(np.abs(raw * scale))
            np.testing.assert_array_equal(mg, (m0 - vel.astype(np.float32)).astype(np.float32))
    print(f"MLP tell ({optimizer}): largest g error / bound {worst:.3f}", flush=True)


def test_mlp_strategy_improves():
    # maximising -MSE: the student moves towards the teacher
    import paper_2212_04180_amd as P
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get("mlp_teacher")
    es = P.ES(cfg)
    log = _np(es.run(30))[:, 0]
    assert log[-5:].mean() > log[:5].mean()


def test_mlp_rejects_fp32_mode():
    import paper_2212_04180_amd as P
    with pytest.raises(P.EsError):
        P.ES(_cfg(mlp_bf16=0))


@pytest.mark.parametrize("strategy,popsize,runs,optimizer", [(0, 1024, 1, 0), (0, 8, 3, 0), (0, 8, 2, 1), (1, 8, 1, 0),
                                                        (0, 4, 1, 0)])
def test_teacher_in_gradient_launch_equals_standalone(strategy, popsize, runs, optimizer):
    """After the first generation the gradient launch also computes the next
    generation's inputs and teacher outputs (OpenAI-ES with Adam or ClipUp;
    PGPE, and workgroups under 256 threads (N = 4), keep the separate teacher
    kernel).  A second handle restored to the same state, whose evaluate
    therefore runs the teacher kernel, gives the same fitness bits: the
    teacher's sums do not depend on the workgroup that runs them."""
    import paper_2212_04180_amd as P
    cfg = _cfg(popsize=popsize, num_runs=runs, strategy=strategy, optimizer=optimizer, sigma_lr=0.2,
               sigma_max_change=0.2, clipup_max_speed=0.05, clipup_momentum=0.9)
    a, b = P.ES(cfg), P.ES(cfg)
    for _ in range(3):
        a.step()
    st = a.get_state()
    b.set_state(st["m"], st["m1"], st["v"], st["t"])
    if strategy == 1:
        b.set_strategy_state(sigma=a.strategy_state()[0])
    if optimizer == 1:
        b.set_strategy_state(velocity=a.strategy_state(sigma=False, velocity=True)[1])
    a.ask()
    fa = a.eval()
    b.ask()
    fb = b.eval()
    assert torch.equal(fa, fb)
    # and the next generation, after a gradient launch on both handles
    a.tell(fa)
    b.tell(fb)
    a.ask()
    b.ask()
    assert torch.equal(a.eval(), b.eval())
