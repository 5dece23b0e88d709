"""The oracle's C code built with AddressSanitizer and UndefinedBehaviorSanitizer
(host only) and driven through every entry point the tests use: every
problem (ragged D, the MLP), every strategy and optimiser, every shaping,
schedules, weight decay, several runs, and non-finite fitness.  Any
out-of-bounds access, use of freed memory, signed overflow, misaligned or
null access or invalid shift in the oracle aborts the child process."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "esoracle.c")

DRIVER = r'''
import math, sys
import numpy as np
sys.path.insert(0, sys.argv[1])
from oracle import oracle as O
def go(T=3, **kw):
    es = O.OracleES(O.OracleConfig(**kw))
    for _ in range(T):
        es.ask()
        f = es.eval() if kw.get("problem", O.PROB_SPHERE) != O.PROB_NONE else None
        if f is None:
            f = np.random.default_rng(0).standard_normal((es.cfg.num_runs, es.cfg.popsize)).astype(np.float32)
            f[0, 0] = np.nan
            f[-1, -1] = np.inf
        es.tell(f)
for prob in (O.PROB_SPHERE, O.PROB_SHIFTED_SPHERE, O.PROB_ROSENBROCK, O.PROB_RASTRIGIN):
    for D in (1, 5, 13):
        go(num_dims=D, popsize=6, num_runs=2, problem=prob)
go(T=2, num_dims=O.MLP_IN * O.MLP_H + O.MLP_H + O.MLP_H * O.MLP_H + O.MLP_H + O.MLP_H * O.MLP_OUT + O.MLP_OUT,
   popsize=2, problem=O.PROB_MLP, maximize=1, init=O.INIT_FANIN_NORMAL, seed=3, mlp_batch=8)
for shaping in (O.SHAPE_CENTERED_RANK, O.SHAPE_RAW, O.SHAPE_Z_SCORE):
    go(num_dims=9, popsize=8, num_runs=3, shaping=shaping, w_decay=0.01, sigma_decay=0.99, sigma_final=0.05,
       lr_decay=0.98, lr_final=0.001, problem=O.PROB_RASTRIGIN)
go(num_dims=7, popsize=10, num_runs=2, problem=O.PROB_NONE)
for strat, opt in ((O.STRAT_PGPE, O.OPT_ADAM), (O.STRAT_PGPE, O.OPT_CLIPUP), (O.STRAT_SNES, O.OPT_ADAM),
                   (O.STRAT_OPENAI_ES, O.OPT_CLIPUP), (O.STRAT_SEP_CMA, O.OPT_ADAM)):
    go(num_dims=11, popsize=8, num_runs=2, strategy=strat, optimizer=opt, problem=O.PROB_ROSENBROCK,
       lr=1.0 if strat == O.STRAT_SNES else 0.01)
print("sanitized oracle ok")
'''


def test_oracle_under_asan_and_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    libasan = subprocess.check_output([gcc, "-print-file-name=libasan.so"], text=True).strip()
    if not os.path.isabs(libasan) or not os.path.exists(libasan):
        pytest.skip("libasan not available")
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.check_call([gcc, "-O1", "-g", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                           "-o", lib, SRC, "-lm"])
    env = dict(os.environ, ESMI_ORACLE_LIB=lib, LD_PRELOAD=libasan,
               ASAN_OPTIONS="detect_leaks=0:exitcode=23", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", DRIVER, ROOT], env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "sanitized oracle ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
