"""Sort-based ranks: populations beyond the 16384 order keys a rank workgroup
holds in LDS (or plan_rank_path 2) take the run's composite keys (key,
member) through a radix sort, a member's position being its rank.  Checked
here (marked gpu):
  - beyond 16384 members, ranks and centered-rank weights bit-exact against
    the oracle's brute-force count (one run: the device-wide sort; several
    runs: the segmented sort), with ties and IEEE specials;
  - at sizes both paths take, three generations of every strategy and
    shaping give the same bits on either path (ranks, weights, state,
    best-so-far), including z-scores, weight decay and PGPE's mean of y,
    which the sort path computes once per run instead of per workgroup;
  - 2^17 members end to end, and 2^24 (the largest accepted) for one
    generation, against numpy's stable argsort of the same keys (the
    oracle's quadratic count is too slow at those sizes).
"""
import numpy as np
import pytest
import torch

from inputs import fitness_with_ties
from oracle import oracle as O

pytestmark = pytest.mark.gpu


def _P():
    import paper_2212_04180_amd as P
    return P


def _cfg(**kw):
    P = _P()
    base = dict(num_dims=24, popsize=64, num_runs=1, sigma=0.1, lr=0.01, seed=11, init=P.INIT_UNIFORM,
                init_lo=-2.0, init_hi=2.0, problem=P.PROB_NONE)
    base.update(kw)
    return P.ESConfig(**base)


def _np(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def _argsort_ranks(f, maximize):
    """Stable ascending ranks of the oracle's keys (NaN the worst, ties by index)."""
    k = -f.astype(np.float64) if maximize else f.astype(np.float64)
    k = np.where(np.isnan(k), np.inf, k)
    order = np.argsort(k, kind="stable")
    r = np.empty(f.shape[0], np.int32)
    r[order] = np.arange(f.shape[0], dtype=np.int32)
    return r


def _centered(rk, N):
    # the fp32 quotient (2 rank - (N - 1)) / (2 (N - 1)) of exact integers
    return (np.float32(2) * rk.astype(np.float32) - np.float32(N - 1)) / np.float32(2 * (N - 1))


@pytest.mark.parametrize("N,R,maximize", [(16386, 1, 0), (20000, 3, 1)])
def test_sort_ranks_match_oracle_beyond_lds(N, R, maximize):
    P = _P()
    es = P.ES(_cfg(popsize=N, num_runs=R, maximize=maximize))
    f = fitness_with_ties(N + R, R, N, ties=True, specials=True)
    es.ask()
    es.tell(torch.tensor(f, device="cuda"))
    y, rk = es.shaped()
    y, rk = _np(y), _np(rk)
    for r in range(R):
        np.testing.assert_array_equal(rk[r], O.ranks(f[r], maximize))
        np.testing.assert_array_equal(y[r], O.shape(f[r], maximize))
    print(f"N={N} R={R}: ranks and weights bit-exact on {R * N} members")


CASES = ["centered", "centered_max", "z_score", "raw_wdecay", "centered_wdecay", "pgpe_raw", "pgpe_z", "snes", "sepcma"]


def _case(name):
    P = _P()
    return {
        "centered": dict(),
        "centered_max": dict(maximize=1),
        "z_score": dict(shaping=P.SHAPE_Z_SCORE),
        "raw_wdecay": dict(shaping=P.SHAPE_RAW, w_decay=0.01),
        "centered_wdecay": dict(w_decay=0.01),
        "pgpe_raw": dict(strategy=P.STRAT_PGPE, shaping=P.SHAPE_RAW),
        "pgpe_z": dict(strategy=P.STRAT_PGPE, shaping=P.SHAPE_Z_SCORE),
        "snes": dict(strategy=P.STRAT_SNES),
        "sepcma": dict(strategy=P.STRAT_SEP_CMA),
    }[name]


def _run(cfg, fits):
    P = _P()
    es = P.ES(cfg)
    out = []
    for f in fits:
        es.ask()
        es.tell(torch.tensor(f, device="cuda"))
        y, rk = es.shaped()
        st = es.get_state()
        bx, bf = es.best()
        rec = [_np(y), _np(rk), _np(st["m"]), _np(st["m1"]), _np(st["v"]), _np(bx), _np(bf)]
        if cfg.strategy in (P.STRAT_PGPE, P.STRAT_SNES, P.STRAT_SEP_CMA):
            rec.append(_np(es.strategy_state(sigma=True)[0]))
        out.append(rec)
    es.close()
    return out


@pytest.mark.parametrize("N,R", [(64, 2), (2050, 1)])
@pytest.mark.parametrize("case", CASES)
def test_sort_path_equals_count_path(case, N, R):
    fits = [fitness_with_ties(100 * g + N + R, R, N, ties=True, specials=(g == 1)) for g in range(3)]
    a = _run(_cfg(popsize=N, num_runs=R, plan_rank_path=1, **_case(case)), fits)
    b = _run(_cfg(popsize=N, num_runs=R, plan_rank_path=2, **_case(case)), fits)
    for g, (ra, rb) in enumerate(zip(a, b)):
        for i, (xa, xb) in enumerate(zip(ra, rb)):
            assert xa.tobytes() == xb.tobytes(), (case, g, i)


def test_large_population_end_to_end():
    """2^17 members, one run: evaluate, sort-based ranks and the update,
    two generations; ranks and weights against a stable argsort of the GPU
    fitness, and the ranks a permutation."""
    P = _P()
    N = 1 << 17
    es = P.ES(_cfg(popsize=N, num_dims=32, problem=P.PROB_SPHERE, seed=4))
    for g in range(2):
        es.ask()
        f = _np(es.eval())
        es.tell(torch.tensor(f, device="cuda"))
        y, rk = es.shaped()
        y, rk = _np(y)[0], _np(rk)[0]
        ref = _argsort_ranks(f[0], 0)
        np.testing.assert_array_equal(rk, ref)
        np.testing.assert_array_equal(np.sort(rk), np.arange(N, dtype=np.int32))
        np.testing.assert_array_equal(y, _centered(ref, N))
    assert es.get_state()["t"] == 2
    print(f"N={N}: two generations, ranks equal to the stable argsort")


def test_largest_population():
    """N = 2^24, the largest accepted population (D = 4, one generation):
    ranks and weights against a stable argsort of the GPU fitness."""
    P = _P()
    N = 1 << 24
    es = P.ES(_cfg(popsize=N, num_dims=4, problem=P.PROB_SPHERE, seed=9))
    es.ask()
    f = _np(es.eval())
    es.tell(torch.tensor(f, device="cuda"))
    y, rk = es.shaped()
    y, rk = _np(y)[0], _np(rk)[0]
    ref = _argsort_ranks(f[0], 0)
    np.testing.assert_array_equal(rk, ref)
    np.testing.assert_array_equal(y, _centered(ref, N))
    assert np.all(np.isfinite(_np(es.get_state()["m"])))
    print(f"N={N}: ranks equal to the stable argsort")
