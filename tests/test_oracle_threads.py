"""The oracle's parallel loops (members, blocks of dimensions) give the same
bits for any thread count: every output's own sum keeps its serial order.
Checked on whole generations of every strategy, with dimension counts that
leave a ragged last block, and on the MLP fitness of a few members."""
import os

import numpy as np
import pytest

from oracle import oracle as O


def _threads():
    return max(2, len(os.sched_getaffinity(0)))


def _run(cfg, gens, nthreads):
    O.set_threads(nthreads)
    try:
        es = O.OracleES(cfg)
        outs = []
        for _ in range(gens):
            out = es.step()
            outs.append((out["fitness"].copy(), out["y"].copy(), out["g"].copy()))
        st = es.get_state()
        return outs, st
    finally:
        O.set_threads(_threads())


@pytest.mark.parametrize("kw", [
    dict(num_dims=10003, popsize=64, num_runs=2, problem=O.PROB_SHIFTED_SPHERE, init=O.INIT_ZERO, sigma=0.01,
         lr=0.001, seed=2),
    dict(num_dims=9001, popsize=16, problem=O.PROB_RASTRIGIN, init_lo=-5.12, init_hi=5.12, sigma=0.2, lr=0.02),
    dict(num_dims=8197, popsize=12, problem=O.PROB_ROSENBROCK, strategy=O.STRAT_PGPE, init_lo=-2.0, init_hi=2.0),
    dict(num_dims=8195, popsize=12, problem=O.PROB_SPHERE, strategy=O.STRAT_SNES, sigma=0.5),
    dict(num_dims=8199, popsize=12, problem=O.PROB_SPHERE, strategy=O.STRAT_SEP_CMA, sigma=0.5),
    dict(num_dims=8192, popsize=10, problem=O.PROB_SPHERE, w_decay=0.1, optimizer=O.OPT_CLIPUP),
])
def test_generations_bit_identical_across_thread_counts(kw):
    cfg = O.OracleConfig(**kw)
    a_out, a_st = _run(cfg, 3, 1)
    b_out, b_st = _run(cfg, 3, _threads())
    for x, y in zip(a_out, b_out):
        for u, v in zip(x, y):
            np.testing.assert_array_equal(u, v)
    for k in a_st:
        np.testing.assert_array_equal(np.asarray(a_st[k]), np.asarray(b_st[k]), err_msg=k)


def test_mlp_fitness_bit_identical_across_thread_counts():
    D = O.mlp_num_params()
    cfg = O.OracleConfig(num_dims=D, popsize=8, problem=O.PROB_MLP, init=O.INIT_FANIN_NORMAL, sigma=0.02,
                         lr=0.01, seed=3, maximize=1)
    m = O.init_mean(cfg, 0)
    pd = O.problem_data(cfg)
    js = np.arange(8, dtype=np.int32)
    O.set_threads(1)
    try:
        f1 = O.eval_members(cfg, 0, 0, m, pd, js)
    finally:
        O.set_threads(_threads())
    f2 = O.eval_members(cfg, 0, 0, m, pd, js)
    np.testing.assert_array_equal(f1, f2)
    assert O.get_threads() == _threads()
