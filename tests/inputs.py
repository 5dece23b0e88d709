"""Seeded synthetic inputs shared by the GPU path and the oracle in tests.

Holds none of the method's arithmetic: only numpy random draws of fitness
vectors and search states with a stated distribution and structure, and the
mapping of a library config onto the oracle's config (field by field).
"""
from __future__ import annotations

import numpy as np

from oracle import oracle as O


def to_oracle(cfg) -> O.OracleConfig:
    """Same hyper-parameters, oracle-side container."""
    keys = ["num_dims", "popsize", "num_runs", "sigma", "lr", "beta1", "beta2", "eps", "maximize", "shaping",
            "seed", "init", "init_lo", "init_hi", "problem", "rastrigin_a", "mlp_batch", "mlp_bf16", "mlp_tanh_out",
            "sigma_decay", "sigma_final", "lr_decay", "lr_final", "w_decay", "strategy", "optimizer", "sigma_lr",
            "sigma_max_change", "clipup_max_speed", "clipup_momentum", "snes_temperature", "elite_ratio"]
    return O.OracleConfig(**{k: getattr(cfg, k) for k in keys})


def fitness_with_ties(seed: int, R: int, N: int, ties: bool = True, specials: bool = False) -> np.ndarray:
    """[R][N] fp32 fitness: normal draws, optionally with runs of equal values
    (values snapped to a coarse grid) and IEEE specials (NaN, +-inf, +-0)."""
    rng = np.random.default_rng(seed)
    f = rng.normal(size=(R, N)) * 3.0
    if ties:
        f = np.round(f * 2.0) / 2.0  # about N/20 distinct values per run
    f = f.astype(np.float32)
    if specials and N >= 8:
        for r in range(R):
            idx = rng.choice(N, size=6, replace=False)
            f[r, idx] = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, np.nan], np.float32)
    return f


def random_state(seed: int, R: int, D: int, t: int):
    """Plausible mid-run Adam state: m ~ U[-3,3], m1 ~ N(0, 0.1^2), v ~ |N(0,1)| * 0.01."""
    rng = np.random.default_rng(seed)
    m = rng.uniform(-3, 3, size=(R, D)).astype(np.float32)
    m1 = (rng.normal(size=(R, D)) * 0.1).astype(np.float32)
    v = (np.abs(rng.normal(size=(R, D))) * 0.01).astype(np.float32)
    return m, m1, v, t
