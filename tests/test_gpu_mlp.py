"""Neuroevolution fitness on the GPU (bf16 matrix cores) against the oracle's
bf16-emulating CPU forward (marked gpu).

Tolerance: |df| <= 2e-2 * |f| (f = -MSE, a sum of non-negative terms).  The
two sides differ by the fp32-vs-fp64 accumulation order, the hardware tanh and
exp against libm, and the bf16 rounding decisions those flip.
"""
import numpy as np
import pytest
import torch

from inputs import to_oracle
from oracle import oracle as O

pytestmark = pytest.mark.gpu

TOL = 2e-2


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
        assert np.all(rel <= TOL), (r, rel)


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
    assert np.all(rel <= TOL), rel
    assert np.all(np.isfinite(f)) and np.all(f < 0)


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
