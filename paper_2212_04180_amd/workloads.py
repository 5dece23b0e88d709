"""Synthetic workloads of the batched OpenAI-ES generation.

Each preset fixes the strategy (App. B tables: OpenAI-ES with Adam and
centered ranks unless stated; PGPE, SNES, ClipUp variants at the D=1e6
geometry) and a benchmark problem (Sec. 3.2: BBOB functions; a
neuroevolution MLP).
The values are plain numbers: no arithmetic of the method lives here.
"""
from __future__ import annotations

from .esmi import (ESConfig, INIT_FANIN_NORMAL, INIT_UNIFORM, INIT_ZERO, OPT_CLIPUP, PROB_MLP, PROB_RASTRIGIN,
                   PROB_ROSENBROCK, PROB_SHIFTED_SPHERE, PROB_SPHERE, STRAT_PGPE, STRAT_SEP_CMA, STRAT_SNES)

# name -> (config, generations)
WORKLOADS = {
    # sphere, D=16, N=32, R=1, sigma 0.1, lr 0.01, mean U[-5,5] seed 0, 100 generations
    "sphere_d16": (ESConfig(num_dims=16, popsize=32, num_runs=1, sigma=0.1, lr=0.01, seed=0,
                            init=INIT_UNIFORM, init_lo=-5.0, init_hi=5.0, problem=PROB_SPHERE), 100),
    # Rosenbrock, D=1000, N=256, R=1, sigma 0.05, lr 0.005, mean U[-2,2] seed 1, 500 generations
    "rosenbrock_d1000": (ESConfig(num_dims=1000, popsize=256, num_runs=1, sigma=0.05, lr=0.005, seed=1,
                                  init=INIT_UNIFORM, init_lo=-2.0, init_hi=2.0, problem=PROB_ROSENBROCK), 500),
    # R=1024 Rastrigin runs (keys 0..1023), D=100, N=64, sigma 0.2, lr 0.02, U[-5.12,5.12], 200 generations
    "rastrigin_r1024": (ESConfig(num_dims=100, popsize=64, num_runs=1024, sigma=0.2, lr=0.02, seed=0,
                                 init=INIT_UNIFORM, init_lo=-5.12, init_hi=5.12, problem=PROB_RASTRIGIN,
                                 rastrigin_a=10.0), 200),
    # shifted sphere, D=1e6, N=2048, R=1, sigma 0.01, lr 0.001, mean 0, s ~ N(0,1) seed 2, 20 generations
    "shifted_sphere_d1m": (ESConfig(num_dims=1_000_000, popsize=2048, num_runs=1, sigma=0.01, lr=0.001, seed=2,
                                    init=INIT_ZERO, problem=PROB_SHIFTED_SPHERE), 20),
    # MLP 64-256-256-16 tanh (D=86544), N=1024, sigma 0.02, lr 0.01, -MSE vs teacher (seed 3), 50 generations
    "mlp_teacher": (ESConfig(num_dims=86544, popsize=1024, num_runs=1, sigma=0.02, lr=0.01, seed=3,
                             init=INIT_FANIN_NORMAL, problem=PROB_MLP, maximize=1, mlp_batch=256, mlp_bf16=1), 50),
    # The other strategies on the D=1e6 shifted sphere (N=2048): PGPE with Adam
    # (App. B PGPE table: sigma learning rate 0.2, max change 0.2), OpenAI-ES
    # with ClipUp, and SNES (App. B SNES table: temperature 12; the standard
    # SNES rates eta_m = 1 and eta_sigma = (3 + ln D) / (5 sqrt D) = 0.00336).
    "pgpe_shifted_sphere_d1m": (ESConfig(num_dims=1_000_000, popsize=2048, num_runs=1, sigma=0.01, lr=0.001,
                                         seed=2, init=INIT_ZERO, problem=PROB_SHIFTED_SPHERE, strategy=STRAT_PGPE,
                                         sigma_lr=0.2, sigma_max_change=0.2), 20),
    "clipup_shifted_sphere_d1m": (ESConfig(num_dims=1_000_000, popsize=2048, num_runs=1, sigma=0.01, lr=0.05,
                                           seed=2, init=INIT_ZERO, problem=PROB_SHIFTED_SPHERE,
                                           optimizer=OPT_CLIPUP, clipup_max_speed=0.1, clipup_momentum=0.9), 20),
    "snes_shifted_sphere_d1m": (ESConfig(num_dims=1_000_000, popsize=2048, num_runs=1, sigma=0.01, lr=1.0,
                                         seed=2, init=INIT_ZERO, problem=PROB_SHIFTED_SPHERE, strategy=STRAT_SNES,
                                         sigma_lr=0.00336, snes_temperature=12.0), 20),
    # Sep-CMA-ES (App. B table: elite ratio 0.5), independent members
    "sepcma_shifted_sphere_d1m": (ESConfig(num_dims=1_000_000, popsize=2048, num_runs=1, sigma=0.01, lr=0.0,
                                           seed=2, init=INIT_ZERO, problem=PROB_SHIFTED_SPHERE,
                                           strategy=STRAT_SEP_CMA, elite_ratio=0.5), 20),
}


def get(name: str) -> tuple[ESConfig, int]:
    cfg, T = WORKLOADS[name]
    return ESConfig(**{k: getattr(cfg, k) for k in cfg.__dataclass_fields__}), T
