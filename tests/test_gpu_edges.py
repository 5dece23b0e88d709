"""Every strategy at tiny and ragged geometries on the GPU (marked gpu),
stage by stage against the oracle.

D of 1, 3, 5 and 9 leave a partial Philox block (and for D < 4 a single one);
N of 2 leaves one antithetic pair, N of 6 an odd pair count.  Bars as in the
per-strategy tests: fitness 1e-5 relative, mean, per-dimension sigma,
velocity, paths and covariance 1e-5 relative, run sigma 1e-5."""
import numpy as np
import pytest
import torch

from inputs import to_oracle
from oracle import oracle as O

pytestmark = pytest.mark.gpu


def _P():
    import paper_2212_04180_amd as P
    return P


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


# name -> (strategy, optimizer)
STRATS = {"openai-adam": (0, 0), "openai-clipup": (0, 1), "pgpe-adam": (1, 0), "pgpe-clipup": (1, 1),
          "snes": (2, 0), "sepcma": (3, 0)}
GEOMS = [(1, 2, 1), (3, 4, 3), (5, 6, 2), (9, 6, 1)]


def _cfg(strategy, optimizer, D, N, R):
    P = _P()
    kw = dict(num_dims=D, popsize=N, num_runs=R, sigma=0.3, lr=0.05, seed=41 + D, init_lo=-2.0, init_hi=2.0,
              problem=P.PROB_ROSENBROCK if D > 1 else P.PROB_RASTRIGIN, strategy=strategy, optimizer=optimizer,
              sigma_lr=0.2, sigma_max_change=0.2, clipup_max_speed=0.2, clipup_momentum=0.9,
              snes_temperature=12.0, elite_ratio=0.5, sigma_decay=0.97, sigma_final=0.05)
    if strategy == P.STRAT_SNES:
        kw.update(lr=1.0, sigma_lr=0.3)
    if strategy == P.STRAT_SEP_CMA:
        kw.update(lr=0.0, sigma_decay=1.0, sigma_final=0.0)
    return P.ESConfig(**kw)


def _rel(a, b, floor):
    a = a.astype(np.float64)
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), floor)))


@pytest.mark.parametrize("geom", GEOMS, ids=lambda g: "D%d-N%d-R%d" % g)
@pytest.mark.parametrize("name", list(STRATS))
def test_tiny_and_ragged_geometries_match_oracle(name, geom):
    P = _P()
    strategy, optimizer = STRATS[name]
    D, N, R = geom
    cfg = _cfg(strategy, optimizer, D, N, R)
    clip = optimizer == P.OPT_CLIPUP and strategy != P.STRAT_SNES
    es = P.ES(cfg)
    ref = O.OracleES(to_oracle(cfg))
    print("case", name, geom, flush=True)
    for t in range(6):
        st = es.get_state()
        sig = vel = None
        if strategy != P.STRAT_OPENAI_ES or clip:
            sg, ve = es.strategy_state(sigma=strategy != P.STRAT_OPENAI_ES, velocity=clip)
            sig = _np(sg) if sg is not None else None
            vel = _np(ve) if ve is not None else None
        ref.set_state(_np(st["m"]), _np(st["m1"]), _np(st["v"]), st["t"], sig=sig, vel=vel)
        ref.set_hparams(*es.get_hparams())
        es.ask()
        f = _np(es.eval())
        fr = ref.eval()
        assert np.all(np.abs(f - fr) <= 1e-5 * np.maximum(np.abs(fr), 1e-30)), (t, f, fr)
        es.tell(torch.tensor(f, device="cuda"))
        ref.tell(f)
        st = es.get_state()
        m = _np(st["m"])
        if strategy == P.STRAT_SEP_CMA:
            assert _rel(m, ref.m, 1e-3) <= 1e-5, t
            w = O.cma_weights(to_oracle(cfg))
            mu_eff = 1.0 / np.sum(w ** 2)
            c_s = (mu_eff + 2.0) / (D + mu_eff + 5.0)
            a_s = np.sqrt(c_s * (2.0 - c_s) * mu_eff)
            dps = np.abs(_np(st["m1"]).astype(np.float64) - ref.m1)
            assert np.all(dps <= a_s * (3e-7 * 5.77 + 8e-7) + 2 * np.spacing(np.abs(ref.m1))), t
            assert _rel(_np(st["v"]), ref.v, 1e-2) <= 1e-5, t
            assert _rel(_np(es.strategy_state()[0]), ref.sig, 1e-6) <= 1e-5, t
        else:
            floor = ref.lr[:, None] * (0.1 if strategy == P.STRAT_SNES else 1.0)
            assert float(np.max(np.abs(m - ref.m) / np.maximum(np.abs(ref.m), floor))) <= 1e-5, t
            if strategy != P.STRAT_OPENAI_ES:
                assert _rel(_np(es.strategy_state()[0]), ref.sig, 1e-30) <= 1e-5, t
            if clip:
                ve = _np(es.strategy_state(sigma=False, velocity=True)[1])
                bound = 1e-5 * max(cfg.clipup_max_speed, float(np.max(np.abs(ref.vel))))
                assert np.max(np.abs(ve - ref.vel)) <= bound, t
        sg, lr = es.get_hparams()
        assert np.all(np.abs(sg - ref.sigma) <= 1e-5 * ref.sigma), t
        np.testing.assert_array_equal(lr, ref.lr)
