"""Python face of the CPU oracle (``esoracle.c``) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  It loads ``liboracle.so`` (plain C, built
with gcc by :func:`build`) through ctypes and never touches the HIP library.

Every function states the passage of the evosax report (arXiv 2212.04180) it
follows; the C file holds the arithmetic and the readings.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "esoracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

PROB_NONE, PROB_SPHERE, PROB_SHIFTED_SPHERE, PROB_ROSENBROCK, PROB_RASTRIGIN, PROB_MLP = range(6)
INIT_UNIFORM, INIT_ZERO, INIT_FANIN_NORMAL = range(3)
SHAPE_CENTERED_RANK, SHAPE_RAW, SHAPE_Z_SCORE = range(3)
STRAT_OPENAI_ES, STRAT_PGPE, STRAT_SNES, STRAT_SEP_CMA = range(4)
OPT_ADAM, OPT_CLIPUP = range(2)
DOM_NOISE, DOM_INIT, DOM_PROBLEM, DOM_EVAL = range(4)
MLP_IN, MLP_H, MLP_OUT = 64, 256, 16


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no fused multiply-add unless written)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
             "-fopenmp", "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("num_dims", ctypes.c_int64),
        ("popsize", ctypes.c_int32),
        ("num_runs", ctypes.c_int32),
        ("sigma", ctypes.c_float),
        ("lr", ctypes.c_float),
        ("beta1", ctypes.c_float),
        ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("maximize", ctypes.c_int32),
        ("shaping", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("init", ctypes.c_int32),
        ("init_lo", ctypes.c_float),
        ("init_hi", ctypes.c_float),
        ("problem", ctypes.c_int32),
        ("rastrigin_a", ctypes.c_float),
        ("mlp_batch", ctypes.c_int32),
        ("mlp_bf16", ctypes.c_int32),
        ("mlp_tanh_out", ctypes.c_int32),
        ("sigma_decay", ctypes.c_float),
        ("sigma_final", ctypes.c_float),
        ("lr_decay", ctypes.c_float),
        ("lr_final", ctypes.c_float),
        ("w_decay", ctypes.c_float),
        ("strategy", ctypes.c_int32),
        ("optimizer", ctypes.c_int32),
        ("sigma_lr", ctypes.c_float),
        ("sigma_max_change", ctypes.c_float),
        ("clipup_max_speed", ctypes.c_float),
        ("clipup_momentum", ctypes.c_float),
        ("snes_temperature", ctypes.c_float),
        ("sigma_vec", ctypes.c_void_p),
        ("elite_ratio", ctypes.c_float),
    ]


@dataclass
class OracleConfig:
    """Hyper-parameters of one batched OpenAI-ES problem (App. B, OpenAI-ES table)."""
    num_dims: int
    popsize: int
    num_runs: int = 1
    sigma: float = 0.1
    lr: float = 0.01
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    maximize: int = 0
    shaping: int = SHAPE_CENTERED_RANK
    seed: int = 0
    init: int = INIT_UNIFORM
    init_lo: float = -5.0
    init_hi: float = 5.0
    problem: int = PROB_SPHERE
    rastrigin_a: float = 10.0
    mlp_batch: int = 256
    mlp_bf16: int = 1
    mlp_tanh_out: int = 0
    # App. B schedules (init = sigma / lr above, then decay and floor per tell)
    sigma_decay: float = 1.0
    sigma_final: float = 0.0
    lr_decay: float = 1.0
    lr_final: float = 0.0
    w_decay: float = 0.0  # weight-decay fitness regularisation (Sec. 3.2)
    # Table 1 strategies beside OpenAI-ES and the ClipUp optimiser (Sec. 3.1);
    # defaults from the App. B PGPE / SNES tables
    strategy: int = STRAT_OPENAI_ES
    optimizer: int = OPT_ADAM
    sigma_lr: float = 0.2
    sigma_max_change: float = 0.2
    clipup_max_speed: float = 0.3
    clipup_momentum: float = 0.9
    snes_temperature: float = 12.0
    elite_ratio: float = 0.5  # Sep-CMA-ES (App. B table)

    def cstruct(self, sigma_vec=None) -> _Cfg:
        c = _Cfg(self.num_dims, self.popsize, self.num_runs, self.sigma, self.lr, self.beta1,
                 self.beta2, self.eps, self.maximize, self.shaping, self.seed, self.init,
                 self.init_lo, self.init_hi, self.problem, self.rastrigin_a, self.mlp_batch,
                 self.mlp_bf16, self.mlp_tanh_out, self.sigma_decay, self.sigma_final,
                 self.lr_decay, self.lr_final, self.w_decay, self.strategy, self.optimizer,
                 self.sigma_lr, self.sigma_max_change, self.clipup_max_speed, self.clipup_momentum,
                 self.snes_temperature, None, self.elite_ratio)
        if sigma_vec is not None:
            c.sigma_vec = sigma_vec.ctypes.data
            c._keep = sigma_vec  # the C side reads through this pointer
        return c


_lib = None


def lib():
    global _lib
    if _lib is None:
        # ESMI_ORACLE_LIB: an alternative build of the same source (the
        # sanitizer test loads one compiled with ASan/UBSan)
        _lib = ctypes.CDLL(os.environ.get("ESMI_ORACLE_LIB") or build())
        P = ctypes.POINTER
        f32, u32, i32, i64, u64 = ctypes.c_float, ctypes.c_uint32, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
        pc = P(_Cfg)
        sig = {
            "or_set_threads": (None, [i32]),
            "or_get_threads": (i32, []),
            "or_philox4x32_10": (None, [u32, u32, P(u32), P(u32)]),
            "or_words": (None, [u64, u32, u32, u32, i64, i64, P(u32)]),
            "or_normals": (None, [u64, u32, u32, u32, i64, i64, P(f32)]),
            "or_mlp_num_params": (i64, []),
            "or_init_mean": (None, [pc, i32, P(f32)]),
            "or_problem_data": (None, [pc, P(f32)]),
            "or_member": (None, [pc, i32, u32, P(f32), i32, P(f32)]),
            "or_population": (None, [pc, i32, u32, P(f32), P(f32)]),
            "or_fitness_bbob": (f32, [i32, P(f32), i64, P(f32), f32]),
            "or_mlp_inputs": (None, [pc, u32, P(f32)]),
            "or_mlp_teacher_out": (None, [pc, P(f32), u32, P(f32)]),
            "or_mlp_fitness": (f32, [pc, P(f32), u32, P(f32)]),
            "or_eval_members": (None, [pc, i32, u32, P(f32), P(f32), P(i32), i32, P(f32)]),
            "or_ranks": (None, [P(f32), i32, i32, P(i32)]),
            "or_shaped_key": (f32, [f32, f32, i32, f32]),
            "or_shape_full": (None, [P(f32), P(f32), i32, i32, i32, f32, P(f32)]),
            "or_penalty": (None, [pc, i32, u32, P(f32), P(f32)]),
            "or_decay": (f32, [f32, f32, f32]),
            "or_noise_sums": (None, [pc, i32, u32, P(f32), P(f32), P(ctypes.c_double), P(ctypes.c_double)]),
            "or_clipup": (None, [pc, f32, P(f32), i64, P(f32), P(f32)]),
            "or_abs_noise_sum": (None, [pc, i32, u32, P(f32), P(ctypes.c_double)]),
            "or_snes_table": (None, [i32, f32, P(f32)]),
            "or_generation_ex": (None, [pc, i32, i64, P(f32), P(f32), P(f32), P(f32), P(f32), P(f32), P(f32),
                                        P(f32), P(f32), P(f32), P(f32), P(ctypes.c_double), P(f32), P(f32)]),
            "or_cma_mu": (i32, [pc]),
            "or_cma_weights": (None, [pc, P(ctypes.c_double)]),
            "or_cma_scale": (None, [i64, f32, P(f32), P(f32)]),
            "or_shape": (None, [P(f32), i32, i32, i32, P(f32)]),
            "or_grad": (None, [pc, i32, u32, P(f32), i64, i64, P(f32)]),
            "or_adam": (None, [pc, i64, P(f32), i64, P(f32), P(f32), P(f32)]),
            "or_generation": (None, [pc, i32, i64, P(f32), P(f32), P(f32), P(f32), P(f32),
                                     P(f32), P(f32), P(f32), P(ctypes.c_double), P(f32), P(f32)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(_lib, name)
            fn.restype = res
            fn.argtypes = args
    return _lib


def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (n <= 0: OpenMP's default, all
    cores).  Results do not depend on it."""
    lib().or_set_threads(int(n))


def get_threads() -> int:
    return int(lib().or_get_threads())


def _p(a, ctype=ctypes.c_float):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# Stage functions (one run at a time).
# --------------------------------------------------------------------------
def philox(key, ctr):
    """Philox-4x32-10 block (Salmon et al., SC'11) for key (k0,k1), counter (c0..c3)."""
    c = (ctypes.c_uint32 * 4)(*[x & 0xFFFFFFFF for x in ctr])
    o = (ctypes.c_uint32 * 4)()
    lib().or_philox4x32_10(key[0] & 0xFFFFFFFF, key[1] & 0xFFFFFFFF, c, o)
    return [o[i] for i in range(4)]


def words(seed, domain, row, t, b0, nb):
    out = np.zeros(4 * nb, dtype=np.uint32)
    lib().or_words(seed, domain, row, t, b0, nb, _p(out, ctypes.c_uint32))
    return out


def normals(seed, domain, row, t, d0, nd):
    """Box-Muller normals of the Gaussian search distribution (Sec. 2.1), dims [d0, d0+nd)."""
    out = np.zeros(nd, dtype=np.float32)
    lib().or_normals(seed, domain, row, t, d0, nd, _p(out))
    return out


def noise(cfg: OracleConfig, run, t, pair, d0=0, nd=None):
    nd = cfg.num_dims - d0 if nd is None else nd
    return normals(cfg.seed + run, DOM_NOISE, pair, t, d0, nd)


def mlp_num_params():
    return int(lib().or_mlp_num_params())


def init_mean(cfg: OracleConfig, run):
    m = np.zeros(cfg.num_dims, dtype=np.float32)
    lib().or_init_mean(cfg.cstruct(), run, _p(m))
    return m


def problem_data(cfg: OracleConfig):
    out = np.zeros(cfg.num_dims, dtype=np.float32)
    lib().or_problem_data(cfg.cstruct(), _p(out))
    return out


def member(cfg, run, t, m, j, sig=None):
    x = np.zeros(cfg.num_dims, dtype=np.float32)
    m = _f32(m)
    lib().or_member(cfg.cstruct(None if sig is None else _f32(sig)), run, t, _p(m), j, _p(x))
    return x


def population(cfg, run, t, m, sig=None):
    """ask (Sec. 2.1): all N members of run ``run`` at generation t, [N][D]."""
    x = np.zeros((cfg.popsize, cfg.num_dims), dtype=np.float32)
    m = _f32(m)
    lib().or_population(cfg.cstruct(None if sig is None else _f32(sig)), run, t, _p(m), _p(x))
    return x


def fitness_bbob(problem, x, s=None, a=10.0):
    x = _f32(x)
    s = _f32(s) if s is not None else None
    return float(lib().or_fitness_bbob(problem, _p(x), x.shape[-1], _p(s), a))


def mlp_inputs(cfg, t):
    X = np.zeros((cfg.mlp_batch, MLP_IN), dtype=np.float32)
    lib().or_mlp_inputs(cfg.cstruct(), t, _p(X))
    return X


def mlp_teacher_out(cfg, teacher, t):
    Y = np.zeros((cfg.mlp_batch, MLP_OUT), dtype=np.float32)
    teacher = _f32(teacher)
    lib().or_mlp_teacher_out(cfg.cstruct(), _p(teacher), t, _p(Y))
    return Y


def mlp_fitness(cfg, x, t, YT):
    x, YT = _f32(x), _f32(YT)
    return float(lib().or_mlp_fitness(cfg.cstruct(), _p(x), t, _p(YT)))


def eval_members(cfg, run, t, m, pdata, js, sig=None):
    """evaluate (Sec. 2.1) for the listed members only."""
    js = np.ascontiguousarray(js, dtype=np.int32)
    f = np.zeros(len(js), dtype=np.float32)
    m = _f32(m)
    pd = _f32(pdata) if pdata is not None else None
    lib().or_eval_members(cfg.cstruct(None if sig is None else _f32(sig)), run, t, _p(m), _p(pd), _p(js, ctypes.c_int32), len(js), _p(f))
    return f


def ranks(f, maximize=0):
    """Stable ascending rank with ties by index (centered-rank shaping, Sec. 3.2)."""
    f = _f32(f)
    r = np.zeros(f.shape[0], dtype=np.int32)
    lib().or_ranks(_p(f), f.shape[0], maximize, _p(r, ctypes.c_int32))
    return r


def shape(f, maximize=0, shaping=SHAPE_CENTERED_RANK):
    f = _f32(f)
    y = np.zeros(f.shape[0], dtype=np.float32)
    lib().or_shape(_p(f), f.shape[0], maximize, shaping, _p(y))
    return y


def shape_full(f, pen=None, maximize=0, shaping=SHAPE_CENTERED_RANK, w_decay=0.0):
    """Fitness shaping with the z-score and weight-decay options of Sec. 3.2
    (readings in ``or_shape_full``); ``pen`` = per-member mean square."""
    f = _f32(f)
    y = np.zeros(f.shape[0], dtype=np.float32)
    pp = _f32(pen) if pen is not None else None
    lib().or_shape_full(_p(f), _p(pp), f.shape[0], maximize, shaping, w_decay, _p(y))
    return y


def penalty(cfg, run, t, m, sig=None):
    """Per-member mean square parameter (1/D) sum_d x_jd^2 of run r at generation t."""
    m = _f32(m)
    pen = np.zeros(cfg.popsize, dtype=np.float32)
    lib().or_penalty(cfg.cstruct(None if sig is None else _f32(sig)), run, t, _p(m), _p(pen))
    return pen


def decay(x, rate, final):
    """One step of the App. B schedule: max(x * rate, final) in fp32."""
    return float(lib().or_decay(x, rate, final))


def noise_sums(cfg, run, t, a, b):
    """A_d = sum_p a_p z_pd and B_d = sum_p b_p (z_pd^2 - 1), fp64."""
    a, b = _f32(a), _f32(b)
    A = np.zeros(cfg.num_dims, np.float64)
    B = np.zeros(cfg.num_dims, np.float64)
    lib().or_noise_sums(cfg.cstruct(), run, t, _p(a), _p(b), _p(A, ctypes.c_double), _p(B, ctypes.c_double))
    return A, B


def abs_noise_sum(cfg, run, t, a):
    """S_d = sum_p |a_p| |z_pd| (fp64): for error bounds of weighted noise sums."""
    a = _f32(a)
    S = np.zeros(cfg.num_dims, np.float64)
    lib().or_abs_noise_sum(cfg.cstruct(), run, t, _p(a), _p(S, ctypes.c_double))
    return S


def clipup(cfg, lr, g, m, vel):
    """One ClipUp step (Toklu et al. 2020) on copies of m and the velocity."""
    g, m, vel = _f32(g), _f32(m).copy(), _f32(vel).copy()
    lib().or_clipup(cfg.cstruct(), lr, _p(g), g.shape[0], _p(m), _p(vel))
    return m, vel


def cma_weights(cfg):
    """Sep-CMA-ES recombination weights by rank (fp64), length mu."""
    mu = int(lib().or_cma_mu(cfg.cstruct()))
    w = np.zeros(mu, np.float64)
    lib().or_cma_weights(cfg.cstruct(), _p(w, ctypes.c_double))
    return w


def cma_scale(D, sigma, C):
    """Sep-CMA-ES sampling scale s_d = fl32(sigma sqrtf(C_d))."""
    s = np.zeros(D, np.float32)
    lib().or_cma_scale(D, float(sigma), _p(_f32(C)), _p(s))
    return s


def snes_table(N, beta):
    """SNES softmax rank utilities indexed by rank' (best = N - 1)."""
    w = np.zeros(N, np.float32)
    lib().or_snes_table(N, beta, _p(w))
    return w


def grad(cfg, run, t, y, d0=0, nd=None):
    """FD gradient estimate g = E^T y / (N sigma) (Sec. 2.1) for dims [d0, d0+nd)."""
    nd = cfg.num_dims - d0 if nd is None else nd
    y = _f32(y)
    g = np.zeros(nd, dtype=np.float32)
    lib().or_grad(cfg.cstruct(), run, t, _p(y), d0, nd, _p(g))
    return g


def adam(cfg, t, g, m, m1, v):
    """Adam step t -> t+1 (Kingma & Ba); returns new (m, m1, v)."""
    g, m, m1, v = _f32(g).copy(), _f32(m).copy(), _f32(m1).copy(), _f32(v).copy()
    lib().or_adam(cfg.cstruct(), t, _p(g), g.shape[0], _p(m), _p(m1), _p(v))
    return m, m1, v


# --------------------------------------------------------------------------
# Whole-strategy view: the ask / evaluate / tell loop of Listing 1, batched
# over R independent seeds (Listing 3).
# --------------------------------------------------------------------------
class OracleES:
    """Batched OpenAI-ES state and loop (Listing 1 / Listing 2 / Listing 3).
    Per-run sigma and learning rate (the vmap over hyper-parameters of
    Sec. 2.2) start from the config and follow the App. B schedules."""

    def __init__(self, cfg: OracleConfig):
        self.cfg = cfg
        R, D = cfg.num_runs, cfg.num_dims
        self.m = np.stack([init_mean(cfg, r) for r in range(R)]) if R else np.zeros((0, D), np.float32)
        self.m1 = np.zeros((R, D), np.float32)
        self.v = np.zeros((R, D), np.float32)
        self.t = 0
        self.pdata = problem_data(cfg) if cfg.problem in (PROB_SHIFTED_SPHERE, PROB_MLP) else None
        self.best_key = np.full(R, math.inf, dtype=np.float64)
        self.best_f = np.full(R, math.nan, dtype=np.float32)
        self.best_x = np.zeros((R, D), np.float32)
        self.sigma = np.full(R, cfg.sigma, dtype=np.float32)
        self.lr = np.full(R, cfg.lr, dtype=np.float32)
        # per-dimension sigma (PGPE, SNES) and ClipUp velocity
        # Sep-CMA-ES keeps its diagonal covariance C (init 1) in sig, p_sigma
        # in m1 and p_c in v
        self.sig = np.full((R, D), 1.0 if cfg.strategy == STRAT_SEP_CMA else cfg.sigma, dtype=np.float32)
        self.vel = np.zeros((R, D), np.float32)

    def set_hparams(self, sigma=None, lr=None):
        if sigma is not None:
            self.sigma = _f32(sigma).copy()
        if lr is not None:
            self.lr = _f32(lr).copy()

    def run_cfg(self, r) -> OracleConfig:
        """The config of run r at the current generation (its sigma and lr)."""
        return replace(self.cfg, sigma=float(self.sigma[r]), lr=float(self.lr[r]))

    def scale(self, r):
        """Sampling scale of run r: sigma vector (PGPE, SNES), sigma sqrt(C) (Sep-CMA-ES)."""
        if self.cfg.strategy == STRAT_SEP_CMA:
            return cma_scale(self.cfg.num_dims, self.sigma[r], self.sig[r])
        return self.sig[r] if self.cfg.strategy != STRAT_OPENAI_ES else None

    def _cs(self, r):
        """C config of run r, with its sampling scale vector where there is one."""
        return self.run_cfg(r).cstruct(self.scale(r))

    def ask(self):
        R, N, D = self.cfg.num_runs, self.cfg.popsize, self.cfg.num_dims
        out = np.zeros((R, N, D), np.float32)
        for r in range(R):
            lib().or_population(self._cs(r), r, self.t, _p(_f32(self.m[r])), _p(out[r]))
        return out

    def eval(self):
        js = np.arange(self.cfg.popsize, dtype=np.int32)
        R, N = self.cfg.num_runs, self.cfg.popsize
        out = np.zeros((R, N), np.float32)
        pd = _f32(self.pdata) if self.pdata is not None else None
        for r in range(R):
            lib().or_eval_members(self._cs(r), r, self.t, _p(_f32(self.m[r])), _p(pd), _p(js, ctypes.c_int32), N,
                                  _p(out[r]))
        return out

    def tell(self, fitness=None):
        """One generation; ``fitness`` [R][N] replaces the built-in evaluation.
        Returns dict of per-run fitness, shaped weights and gradient."""
        cfg = self.cfg
        R, N, D = cfg.num_runs, cfg.popsize, cfg.num_dims
        out_f = np.zeros((R, N), np.float32)
        out_y = np.zeros((R, N), np.float32)
        out_g = np.zeros((R, D), np.float32)
        pd = _f32(self.pdata) if self.pdata is not None else None
        for r in range(R):
            c = self.run_cfg(r).cstruct()
            m, m1, v = self.m[r].copy(), self.m1[r].copy(), self.v[r].copy()
            vel, sig = self.vel[r].copy(), self.sig[r].copy()
            fin = _f32(fitness[r]) if fitness is not None else None
            bk = ctypes.c_double(self.best_key[r])
            bf = np.array([self.best_f[r]], np.float32)
            bx = self.best_x[r].copy()
            fo, yo, go = np.zeros(N, np.float32), np.zeros(N, np.float32), np.zeros(D, np.float32)
            so = np.array([self.sigma[r]], np.float32)
            lib().or_generation_ex(c, r, self.t, _p(pd), _p(m), _p(m1), _p(v), _p(vel), _p(sig), _p(so), _p(fin),
                                   _p(fo), _p(yo), _p(go), ctypes.byref(bk), _p(bf), _p(bx))
            if cfg.strategy == STRAT_SEP_CMA:
                self.sigma[r] = so[0]
            self.m[r], self.m1[r], self.v[r] = m, m1, v
            self.vel[r], self.sig[r] = vel, sig
            self.best_key[r], self.best_f[r], self.best_x[r] = bk.value, bf[0], bx
            out_f[r], out_y[r], out_g[r] = fo, yo, go
            if cfg.strategy == STRAT_OPENAI_ES:
                self.sigma[r] = decay(float(self.sigma[r]), cfg.sigma_decay, cfg.sigma_final)
            # (Sep-CMA-ES adapts sigma by path length instead of a schedule)
            self.lr[r] = decay(float(self.lr[r]), cfg.lr_decay, cfg.lr_final)
        self.t += 1
        return {"fitness": out_f, "y": out_y, "g": out_g}

    def step(self):
        return self.tell(None)

    def run(self, T):
        """T generations (Listing 2); returns per-generation best fitness [T][R]."""
        log = np.zeros((T, self.cfg.num_runs), np.float32)
        for i in range(T):
            out = self.step()
            f = out["fitness"]
            for r in range(self.cfg.num_runs):
                rk = ranks(f[r], self.cfg.maximize)
                log[i, r] = f[r][int(np.argmin(rk))]
        return log

    def get_state(self):
        return {"m": self.m.copy(), "m1": self.m1.copy(), "v": self.v.copy(), "t": self.t,
                "sigma": self.sigma.copy(), "lr": self.lr.copy(), "sig": self.sig.copy(), "vel": self.vel.copy()}

    def set_state(self, m, m1, v, t, sig=None, vel=None):
        self.m, self.m1, self.v = _f32(m).copy(), _f32(m1).copy(), _f32(v).copy()
        self.t = int(t)
        if sig is not None:
            self.sig = _f32(sig).copy()
        if vel is not None:
            self.vel = _f32(vel).copy()
