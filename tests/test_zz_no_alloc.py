"""es_eval_noalloc, the allocation-free evaluate (marked gpu): the same
fitness bits as es_eval of a handle with the same config, mean, sigma and
generation, on two calls in a row (the second with a smaller input), and a
clear error when the partial sums would not fit the static scratch."""
import dataclasses

import pytest
import torch

pytestmark = pytest.mark.gpu


def _P():
    import paper_2212_04180_amd as P
    return P


def _handle_and_noalloc(cfg, gens):
    P = _P()
    es = P.ES(cfg)
    for _ in range(gens):
        es.step()
    st = es.get_state()
    sigma = torch.tensor(es.get_hparams()[0], device="cuda")
    pdata = es.problem_data() if cfg.problem == P.PROB_SHIFTED_SPHERE else None
    es.ask()
    f_ref = es.eval()
    f = P.eval_noalloc(cfg, st["m"], sigma, st["t"], problem_data=pdata)
    torch.cuda.synchronize()
    return f, f_ref


def test_noalloc_equals_es_eval_twice_then_smaller():
    P = _P()
    big = P.ESConfig(num_dims=1000, popsize=256, num_runs=3, sigma=0.05, lr=0.01, seed=4, init=P.INIT_ZERO,
                     problem=P.PROB_SHIFTED_SPHERE)
    small = P.ESConfig(num_dims=101, popsize=34, num_runs=1, sigma=0.2, lr=0.02, seed=9, init_lo=-5.12,
                       init_hi=5.12, problem=P.PROB_RASTRIGIN)
    for cfg, gens in ((big, 2), (small, 3)):
        print("es_eval_noalloc", cfg.problem, cfg.num_dims, cfg.popsize, cfg.num_runs, flush=True)
        f, f_ref = _handle_and_noalloc(cfg, gens)
        assert torch.isfinite(f_ref).all()
        assert torch.equal(f, f_ref)


def test_noalloc_full_size_equals_es_eval():
    """The D = 1e6, N = 2048 evaluate (12.6 MB of partial sums), then a
    smaller Rosenbrock evaluate on the same scratch."""
    P = _P()
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get("shifted_sphere_d1m")
    print("es_eval_noalloc full size", flush=True)
    f, f_ref = _handle_and_noalloc(cfg, 1)
    assert torch.equal(f, f_ref)
    cfg, _ = workloads.get("rosenbrock_d1000")
    f, f_ref = _handle_and_noalloc(cfg, 2)
    assert torch.equal(f, f_ref)


def test_noalloc_rejects_what_does_not_fit():
    P = _P()
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get("shifted_sphere_d1m")
    cfg = dataclasses.replace(cfg, plan_eval_blocks=4)  # 62,500 chunks of partial sums: 512 MB
    m = torch.zeros(1, cfg.num_dims, device="cuda")
    s = torch.zeros(cfg.num_dims, device="cuda")
    sigma = torch.full((1,), cfg.sigma, device="cuda")
    with pytest.raises(P.EsError, match="static scratch"):
        P.eval_noalloc(cfg, m, sigma, 0, problem_data=s)
    mlp, _ = workloads.get("mlp_teacher")
    with pytest.raises(P.EsError, match="benchmark problems"):
        P.eval_noalloc(mlp, torch.zeros(1, mlp.num_dims, device="cuda"), sigma, 0)
    ragged = P.ESConfig(num_dims=10, popsize=4, num_runs=2, problem=P.PROB_SPHERE)
    with pytest.raises(P.EsError, match="num_dims % 4"):
        P.eval_noalloc(ragged, torch.zeros(2, 10, device="cuda"), torch.ones(2, device="cuda"), 0)
