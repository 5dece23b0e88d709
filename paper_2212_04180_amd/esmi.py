"""ctypes binding of libesmi.so (declared in include/esmi.h).

Argument marshalling only: every step of the generation runs in the HIP
kernels behind the C-ABI.  PyTorch supplies device memory (``tensor.data_ptr``)
and the stream (``torch.cuda.current_stream().cuda_stream``).  There is no
CPU fallback: a missing or unloadable library raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, fields

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libesmi.so")

ES_OK, ES_ERR_ARG, ES_ERR_SEQUENCE, ES_ERR_HIP, ES_ERR_OOM, ES_ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
SHAPE_CENTERED_RANK, SHAPE_RAW, SHAPE_Z_SCORE = 0, 1, 2
PROB_NONE, PROB_SPHERE, PROB_SHIFTED_SPHERE, PROB_ROSENBROCK, PROB_RASTRIGIN, PROB_MLP = range(6)
INIT_UNIFORM, INIT_ZERO, INIT_FANIN_NORMAL = range(3)
FLAG_KEEP_GRAD = 1
STRAT_OPENAI_ES, STRAT_PGPE, STRAT_SNES, STRAT_SEP_CMA = range(4)
OPT_ADAM, OPT_CLIPUP = range(2)

# Every symbol include/esmi.h declares, in declaration order.
EXPORTS = ("es_init", "es_ask", "es_eval", "es_eval_timed", "es_eval_noalloc", "es_tell", "es_run", "es_get_state", "es_set_state",
           "es_get_best", "es_get_shaped", "es_get_grad", "es_set_hparams", "es_get_hparams",
           "es_get_strategy_state", "es_set_strategy_state", "es_get_penalty",
           "es_get_problem_data", "es_debug_noise",
           "es_save_state", "es_load_state", "es_sync", "es_generation", "es_run_path", "es_last_error",
           "es_status_string", "es_destroy")


class EsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [
        ("num_dims", ctypes.c_int64),
        ("seed", ctypes.c_uint64),
        ("popsize", ctypes.c_int32),
        ("num_runs", ctypes.c_int32),
        ("sigma", ctypes.c_float),
        ("lr", ctypes.c_float),
        ("beta1", ctypes.c_float),
        ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("maximize", ctypes.c_int32),
        ("shaping", ctypes.c_int32),
        ("init", ctypes.c_int32),
        ("init_lo", ctypes.c_float),
        ("init_hi", ctypes.c_float),
        ("problem", ctypes.c_int32),
        ("rastrigin_a", ctypes.c_float),
        ("mlp_batch", ctypes.c_int32),
        ("mlp_bf16", ctypes.c_int32),
        ("mlp_tanh_out", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
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
        ("elite_ratio", ctypes.c_float),
        ("plan_eval_blocks", ctypes.c_int32),
        ("plan_tell_split", ctypes.c_int32),
        ("plan_run_path", ctypes.c_int32),
        ("plan_rank_path", ctypes.c_int32),
        ("plan_grid_workgroups", ctypes.c_int32),
        ("plan_grid_spin_limit", ctypes.c_int32),
        ("plan_grid_pack", ctypes.c_int32),
    ]


@dataclass
class ESConfig:
    """Strategy parameters (Listing 1 ``default_params``; App. B OpenAI-ES table)."""
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
    flags: int = 0
    # App. B schedules: after each tell x <- max(x * decay, final)
    sigma_decay: float = 1.0
    sigma_final: float = 0.0
    lr_decay: float = 1.0
    lr_final: float = 0.0
    w_decay: float = 0.0  # weight-decay fitness regularisation (Sec. 3.2)
    # Table 1 strategy and the mean's optimiser; App. B PGPE / SNES defaults
    strategy: int = STRAT_OPENAI_ES
    optimizer: int = OPT_ADAM
    sigma_lr: float = 0.2
    sigma_max_change: float = 0.2
    clipup_max_speed: float = 0.3
    clipup_momentum: float = 0.9
    snes_temperature: float = 12.0
    elite_ratio: float = 0.5  # Sep-CMA-ES (App. B table)
    # launch plan, 0 = the library's choice (esmi.h): evaluate chunk length and
    # gradient split change the summation order; run path 1 per-call, 2 fused,
    # 3 grid loop; rank path 1 counted in LDS (N <= 16384), 2 radix-sorted
    # (same ranks); grid spin limit: polls before a grid-loop wait gives up
    # (-1: at once, the failure path)
    plan_eval_blocks: int = 0
    plan_tell_split: int = 0
    plan_run_path: int = 0
    plan_rank_path: int = 0
    plan_grid_workgroups: int = 0
    plan_grid_spin_limit: int = 0
    plan_grid_pack: int = 0

    def cstruct(self) -> _Config:
        c = _Config()
        for f in fields(self):
            setattr(c, f.name, getattr(self, f.name))
        return c


_lib = None


def lib() -> ctypes.CDLL:
    """Load libesmi.so (built by ``paper_2212_04180_amd.build``); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build the HIP library first "
                           "(python -c 'import __graft_entry__ as g; g.build()')")
    L = ctypes.CDLL(LIB_PATH)
    P, vp = ctypes.POINTER, ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    sig = {
        "es_init": (i32, [P(_Config), vp, P(vp)]),
        "es_ask": (i32, [vp, vp]),
        "es_eval": (i32, [vp, vp]),
        "es_eval_timed": (i32, [vp, vp, vp, vp]),
        "es_eval_noalloc": (i32, [P(_Config), vp, vp, vp, i64, vp, vp]),
        "es_tell": (i32, [vp, vp]),
        "es_run": (i32, [vp, i32, vp]),
        "es_get_state": (i32, [vp, vp, vp, vp, P(i64)]),
        "es_set_state": (i32, [vp, vp, vp, vp, i64]),
        "es_get_best": (i32, [vp, vp, vp]),
        "es_get_shaped": (i32, [vp, vp, vp]),
        "es_get_grad": (i32, [vp, vp]),
        "es_set_hparams": (i32, [vp, vp, vp]),
        "es_get_hparams": (i32, [vp, vp, vp]),
        "es_get_penalty": (i32, [vp, vp]),
        "es_get_strategy_state": (i32, [vp, vp, vp]),
        "es_set_strategy_state": (i32, [vp, vp, vp]),
        "es_get_problem_data": (i32, [vp, vp]),
        "es_debug_noise": (i32, [vp, i32, i64, i32, vp, vp]),
        "es_save_state": (i32, [vp, vp, P(ctypes.c_size_t)]),
        "es_load_state": (i32, [vp, vp, ctypes.c_size_t]),
        "es_sync": (i32, [vp]),
        "es_generation": (i64, [vp]),
        "es_run_path": (i32, [vp, vp]),
        "es_last_error": (ctypes.c_char_p, [vp]),
        "es_status_string": (ctypes.c_char_p, [i32]),
        "es_destroy": (None, [vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype, fn.argtypes = res, args
    _lib = L
    return L


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device tensor expected")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor expected")
    return ctypes.c_void_p(t.data_ptr())


def eval_noalloc(cfg: ESConfig, mean, sigma, t: int, problem_data=None, out=None, stream=None):
    """es_eval_noalloc: the fused sample + evaluate of generation t without a
    handle and without device allocation inside the library.  mean [R][D],
    sigma [R], problem_data [D] or None, out [R][N]: device tensors."""
    if out is None:
        out = torch.empty(cfg.num_runs, cfg.popsize, dtype=torch.float32, device=mean.device)
    st = stream if stream is not None else torch.cuda.current_stream(mean.device)
    cs = cfg.cstruct()
    rc = lib().es_eval_noalloc(ctypes.byref(cs), _ptr(mean), _ptr(problem_data), _ptr(sigma), int(t), _ptr(out),
                               ctypes.c_void_p(st.cuda_stream))
    if rc != ES_OK:
        raise EsError(rc, lib().es_last_error(None).decode())
    return out


class ES:
    """One batched OpenAI-ES strategy living on a GPU (handle of the C-ABI)."""

    def __init__(self, cfg: ESConfig, device: str | torch.device = "cuda:0", stream=None):
        self.cfg = cfg
        self.device = torch.device(device)
        if self.device.type != "cuda":
            raise ValueError("ES runs on a GPU device only")
        torch.cuda.set_device(self.device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self._h = ctypes.c_void_p()
        self._cs = cfg.cstruct()
        st = lib().es_init(ctypes.byref(self._cs), ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(self._h))
        if st != ES_OK:
            raise EsError(st, lib().es_last_error(None).decode())

    # -- helpers -----------------------------------------------------------
    def _check(self, st):
        if st != ES_OK:
            raise EsError(st, lib().es_last_error(self._h).decode())

    def _empty(self, *shape, dtype=torch.float32):
        return torch.empty(*shape, dtype=dtype, device=self.device)

    @property
    def R(self):
        return self.cfg.num_runs

    @property
    def N(self):
        return self.cfg.popsize

    @property
    def D(self):
        return self.cfg.num_dims

    @property
    def t(self) -> int:
        return int(lib().es_generation(self._h))

    @property
    def run_path(self) -> int:
        """The path es_run takes: 1 per-call kernels, 2 fused loop, 3 grid loop."""
        return int(lib().es_run_path(self._h, None))

    @property
    def run_keeps_normals(self) -> bool:
        """Whether es_run's gradient reads the normals its evaluate kept in LDS."""
        k = ctypes.c_int32(0)
        lib().es_run_path(self._h, ctypes.byref(k))
        return bool(k.value)

    # -- ask / evaluate / tell ---------------------------------------------
    def ask(self, materialize: bool = False):
        x = self._empty(self.R, self.N, self.D) if materialize else None
        self._check(lib().es_ask(self._h, _ptr(x)))
        return x

    def eval(self, out=None, events=None):
        """Fitness of the asked population.  events: None, or a (start, stop)
        pair of timing torch.cuda.Event objects, each recorded once before so
        that it exists, which the evaluate kernels then record themselves
        (es_eval_timed)."""
        out = self._empty(self.R, self.N) if out is None else out
        if events is None:
            self._check(lib().es_eval(self._h, _ptr(out)))
            return out
        hs, he = (int(e.cuda_event) for e in events)
        if not hs or not he:
            raise ValueError("es_eval_timed takes created events: record each one once beforehand")
        self._check(lib().es_eval_timed(self._h, _ptr(out), ctypes.c_void_p(hs), ctypes.c_void_p(he)))
        return out

    def tell(self, fitness):
        assert fitness.shape == (self.R, self.N) and fitness.dtype == torch.float32
        self._check(lib().es_tell(self._h, _ptr(fitness)))

    def step(self, fit=None):
        """One generation with the built-in problem; returns the fitness tensor."""
        self.ask()
        f = self.eval(fit)
        self.tell(f)
        return f

    def run(self, T: int, log: bool = True):
        out = self._empty(T, self.R) if (log and T > 0) else None
        self._check(lib().es_run(self._h, int(T), _ptr(out)))
        return out

    # -- state -------------------------------------------------------------
    def get_state(self):
        m, m1, v = (self._empty(self.R, self.D) for _ in range(3))
        t = ctypes.c_int64()
        self._check(lib().es_get_state(self._h, _ptr(m), _ptr(m1), _ptr(v), ctypes.byref(t)))
        return {"m": m, "m1": m1, "v": v, "t": int(t.value)}

    def set_state(self, m, m1, v, t):
        self._check(lib().es_set_state(self._h, _ptr(m), _ptr(m1), _ptr(v), int(t)))

    def best(self):
        x, f = self._empty(self.R, self.D), self._empty(self.R)
        self._check(lib().es_get_best(self._h, _ptr(x), _ptr(f)))
        return x, f

    def shaped(self):
        y = self._empty(self.R, self.N)
        rk = self._empty(self.R, self.N, dtype=torch.int32)
        self._check(lib().es_get_shaped(self._h, _ptr(y), _ptr(rk)))
        return y, rk

    def grad(self):
        g = self._empty(self.R, self.D)
        self._check(lib().es_get_grad(self._h, _ptr(g)))
        return g

    def set_hparams(self, sigma=None, lr=None):
        """Per-run sigma and learning rate of the next generation (host arrays [R])."""
        import numpy as np
        bufs = []
        for a in (sigma, lr):
            if a is None:
                bufs.append(None)
            else:
                b = np.ascontiguousarray(np.asarray(a, dtype=np.float32).reshape(self.R))
                bufs.append(b)
        ptr = [None if b is None else ctypes.c_void_p(b.ctypes.data) for b in bufs]
        self._check(lib().es_set_hparams(self._h, ptr[0], ptr[1]))

    def get_hparams(self):
        import numpy as np
        sg, lr = np.zeros(self.R, np.float32), np.zeros(self.R, np.float32)
        self._check(lib().es_get_hparams(self._h, ctypes.c_void_p(sg.ctypes.data), ctypes.c_void_p(lr.ctypes.data)))
        return sg, lr

    def strategy_state(self, sigma=True, velocity=False):
        """Per-dimension sigma (PGPE, SNES) and/or ClipUp velocity, [R][D] each."""
        sg = self._empty(self.R, self.D) if sigma else None
        ve = self._empty(self.R, self.D) if velocity else None
        self._check(lib().es_get_strategy_state(self._h, _ptr(sg), _ptr(ve)))
        return sg, ve

    def set_strategy_state(self, sigma=None, velocity=None):
        self._check(lib().es_set_strategy_state(self._h, _ptr(sigma), _ptr(velocity)))

    def penalty(self):
        out = self._empty(self.R, self.N)
        self._check(lib().es_get_penalty(self._h, _ptr(out)))
        return out

    def problem_data(self):
        out = self._empty(self.D)
        self._check(lib().es_get_problem_data(self._h, _ptr(out)))
        return out

    def debug_noise(self, run: int, t: int, pair: int):
        nb = (self.D + 3) // 4
        w = self._empty(4 * nb, dtype=torch.int32)
        e = self._empty(self.D)
        self._check(lib().es_debug_noise(self._h, run, t, pair, _ptr(w), _ptr(e)))
        return w, e

    def save(self) -> bytes:
        n = ctypes.c_size_t(0)
        self._check(lib().es_save_state(self._h, None, ctypes.byref(n)))
        buf = ctypes.create_string_buffer(n.value)
        self._check(lib().es_save_state(self._h, buf, ctypes.byref(n)))
        return buf.raw[:n.value]

    def load(self, blob: bytes):
        buf = ctypes.create_string_buffer(blob, len(blob))
        self._check(lib().es_load_state(self._h, buf, len(blob)))

    def sync(self):
        self._check(lib().es_sync(self._h))

    def close(self):
        if self._h:
            lib().es_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
