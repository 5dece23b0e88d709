"""Pins of the oracle's neuroevolution fitness: a 64-256-256-16 tanh MLP
(network definitions and parameter reshaping, Sec. 3.2) scored by -MSE against
a fixed random teacher, checked against torch on the CPU."""
import numpy as np
import pytest
import torch

from oracle import oracle as O

SHAPES = [(256, 64), (256, 256), (16, 256)]


def _cfg(**kw):
    base = dict(num_dims=86544, popsize=4, sigma=0.02, lr=0.01, seed=3, init=O.INIT_FANIN_NORMAL,
                problem=O.PROB_MLP, maximize=1, mlp_batch=256, mlp_bf16=1)
    base.update(kw)
    return O.OracleConfig(**base)


def _unflatten(p):
    out, off = [], 0
    for fo, fi in SHAPES:
        W = p[off:off + fo * fi].reshape(fo, fi)
        off += fo * fi
        b = p[off:off + fo]
        off += fo
        out.append((W, b))
    assert off == p.shape[0]
    return out


def _bf16(a):
    return torch.tensor(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float32).double()


def _torch_forward(p, X, bf16, tanh_out=False):
    h = _bf16(X) if bf16 else torch.tensor(X).double()
    layers = _unflatten(p)
    for i, (W, b) in enumerate(layers):
        Wt = _bf16(W) if bf16 else torch.tensor(W).double()
        pre = (h @ Wt.T + torch.tensor(b).double()).float().double()
        if i < 2 or tanh_out:
            h = torch.tanh(pre).float()
            if i < 2 and bf16:
                h = h.to(torch.bfloat16).to(torch.float32)
            h = h.double()
        else:
            h = pre
    return h.float().numpy()


def test_param_count_and_layout():
    assert O.mlp_num_params() == 64 * 256 + 256 + 256 * 256 + 256 + 256 * 16 + 16 == 86544
    cfg = _cfg()
    m = O.init_mean(cfg, 0)
    layers = _unflatten(m)
    for (W, b), (fo, fi) in zip(layers, SHAPES):
        assert np.all(b == 0)
        # N(0, 1/fan_in) weights: the empirical std matches 1/sqrt(fan_in)
        assert W.std() == pytest.approx(1 / np.sqrt(fi), rel=0.05)
        assert abs(W.mean()) < 5 / np.sqrt(fi) / np.sqrt(W.size)


@pytest.mark.parametrize("bf16", [0, 1])
def test_forward_matches_torch(bf16):
    cfg = _cfg(mlp_bf16=bf16)
    teacher = O.problem_data(cfg)
    t = 2
    X = O.mlp_inputs(cfg, t)
    assert X.shape == (256, 64)
    YT = O.mlp_teacher_out(cfg, teacher, t)
    np.testing.assert_allclose(YT, _torch_forward(teacher, X, False), rtol=0, atol=1e-6)
    m = O.init_mean(cfg, 0)
    x = O.member(cfg, 0, t, m, 1)
    f = O.mlp_fitness(cfg, x, t, YT)
    Y = _torch_forward(x, X, bf16)
    mse = np.mean((Y.astype(np.float64) - YT.astype(np.float64)) ** 2)
    assert f < 0
    assert -f == pytest.approx(mse, rel=1e-5)


def test_student_equal_to_teacher_scores_zero():
    cfg = _cfg(mlp_bf16=0, sigma=0.0)
    teacher = O.problem_data(cfg)
    f = O.eval_members(cfg, 0, 0, teacher, teacher, [0, 3])
    assert np.all(f == 0.0)
    # with bf16 operands the same network is close but not exact
    cfgb = _cfg(mlp_bf16=1, sigma=0.0)
    fb = O.eval_members(cfgb, 0, 0, teacher, teacher, [0])
    assert -1e-3 < fb[0] < 0


def test_inputs_change_per_generation():
    cfg = _cfg()
    X0, X1 = O.mlp_inputs(cfg, 0), O.mlp_inputs(cfg, 1)
    assert abs(np.corrcoef(X0.ravel(), X1.ravel())[0, 1]) < 0.05
    assert X0.std() == pytest.approx(1.0, rel=0.05)
