"""Every strategy at tiny and ragged geometries on the GPU (marked gpu),
stage by stage against the oracle.

D of 1, 3, 5 and 9 leave a partial Philox block (and for D < 4 a single one);
N of 2 leaves one antithetic pair, N of 6 an odd pair count.  Bars as in the
per-strategy tests: fitness 1e-5 relative, mean, per-dimension sigma,
velocity, paths and covariance 1e-5 relative, run sigma 1e-5."""
import dataclasses
import pytest

import stagecheck

pytestmark = pytest.mark.gpu


def _P():
    import paper_2212_04180_amd as P
    return P


# name -> (strategy, optimizer)
STRATS = {"openai-adam": (0, 0), "openai-clipup": (0, 1), "pgpe-adam": (1, 0), "pgpe-clipup": (1, 1),
          "snes": (2, 0), "sepcma": (3, 0)}
GEOMS = [(1, 2, 1), (3, 4, 3), (5, 6, 2), (9, 6, 1)]


def _cfg(strategy, optimizer, D, N, R):
    P = _P()
    kw = dict(num_dims=D, popsize=N, num_runs=R, sigma=0.3, lr=0.05, seed=41 + D, init_lo=-2.0, init_hi=2.0,
              problem=P.PROB_ROSENBROCK if D > 1 else P.PROB_RASTRIGIN, strategy=strategy, optimizer=optimizer,
              sigma_lr=0.2, sigma_max_change=0.2, clipup_max_speed=0.2, clipup_momentum=0.9,
              snes_temperature=12.0, elite_ratio=0.5, sigma_decay=0.97, sigma_final=0.05,
              flags=P.FLAG_KEEP_GRAD)
    if strategy == P.STRAT_SNES:
        kw.update(lr=1.0, sigma_lr=0.3)
    if strategy == P.STRAT_SEP_CMA:
        kw.update(lr=0.0, sigma_decay=1.0, sigma_final=0.0)
    return P.ESConfig(**kw)


@pytest.mark.parametrize("geom", GEOMS, ids=lambda g: "D%d-N%d-R%d" % g)
@pytest.mark.parametrize("name", list(STRATS))
def test_tiny_and_ragged_geometries_match_oracle(name, geom):
    P = _P()
    strategy, optimizer = STRATS[name]
    print("case", name, geom, flush=True)
    stagecheck.run(P, _cfg(strategy, optimizer, *geom), 6)


def test_largest_run_count_fused_and_per_call():
    """num_runs = 65535, the largest accepted (runs are the y dimension of the
    per-call grids): es_run through the fused loop (one workgroup per run) and
    through the per-call kernels gives the same bits, and sampled runs score
    as standalone oracle runs with key seed + r."""
    import dataclasses

    import numpy as np
    import torch

    from inputs import to_oracle
    from oracle import oracle as O
    P = _P()
    cfg = P.ESConfig(num_dims=5, popsize=2, num_runs=65535, sigma=0.3, lr=0.05, seed=0, init_lo=-2.0, init_hi=2.0,
                     problem=P.PROB_ROSENBROCK)
    out = {}
    for path in ("1", "2"):
        es = P.ES(dataclasses.replace(cfg, plan_run_path=int(path)))
        log = es.run(3)
        st = es.get_state()
        torch.cuda.synchronize()
        out[path] = [t.cpu().numpy() for t in (log, st["m"], st["m1"], st["v"])]
    for a, b in zip(out["1"], out["2"]):
        np.testing.assert_array_equal(a, b)
    es = P.ES(cfg)
    es.ask()
    f = es.eval()
    torch.cuda.synchronize()
    f = f.cpu().numpy()
    for r in (0, 1, 40000, 65534):
        oc = dataclasses.replace(to_oracle(cfg), num_runs=1, seed=r)
        fr = O.OracleES(oc).eval()[0]
        assert np.all(np.abs(f[r] - fr) <= 1e-5 * np.abs(fr)), (r, f[r], fr)


@pytest.mark.parametrize("N", [16384, 16386])
@pytest.mark.parametrize("name", list(STRATS))
def test_largest_population_matches_oracle(name, N):
    """N = 16384 with the ranks counted in LDS (the keys fill 64 KB; the
    library itself would sort at this size), and N = 16386, the smallest that
    must take the sort-based ranks; D = 37 (ragged), two runs, stage by stage."""
    import dataclasses
    P = _P()
    strategy, optimizer = STRATS[name]
    cfg = _cfg(strategy, optimizer, 37, N, 2)
    if N <= 16384:
        cfg = dataclasses.replace(cfg, plan_rank_path=1)
    print("case", name, N, flush=True)
    stagecheck.run(P, cfg, 2)
