"""MI355X-native batched ES generations (ask / evaluate / tell): OpenAI-ES, PGPE,
SNES and Sep-CMA-ES.

The hot path is the HIP library ``libesmi.so`` (C-ABI in ``include/esmi.h``);
this package is its thin Python binding and the synthetic workload presets.
"""
from .esmi import (ES, ESConfig, EsError, FLAG_KEEP_GRAD, INIT_FANIN_NORMAL, INIT_UNIFORM, INIT_ZERO,
                   PROB_MLP, PROB_NONE, PROB_RASTRIGIN, PROB_ROSENBROCK, PROB_SHIFTED_SPHERE, PROB_SPHERE,
                   SHAPE_CENTERED_RANK, SHAPE_RAW, SHAPE_Z_SCORE, STRAT_OPENAI_ES, STRAT_PGPE, STRAT_SNES, STRAT_SEP_CMA,
                   OPT_ADAM, OPT_CLIPUP, eval_noalloc, lib)

__all__ = ["ES", "ESConfig", "EsError", "lib", "FLAG_KEEP_GRAD", "INIT_FANIN_NORMAL", "INIT_UNIFORM",
           "INIT_ZERO", "PROB_MLP", "PROB_NONE", "PROB_RASTRIGIN", "PROB_ROSENBROCK", "PROB_SHIFTED_SPHERE",
           "PROB_SPHERE", "SHAPE_CENTERED_RANK", "SHAPE_RAW", "SHAPE_Z_SCORE", "STRAT_OPENAI_ES", "STRAT_PGPE",
           "STRAT_SNES", "STRAT_SEP_CMA", "OPT_ADAM", "OPT_CLIPUP"]
