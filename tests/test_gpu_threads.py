"""Handles driven from several host threads at once (marked gpu): each thread
owns a handle on its own stream (per-call generations, es_run's fused loop and
its grid loop), and every result equals the same handle run alone; the error
of a refused es_init stays with the thread that made the call."""
import ctypes
import threading

import pytest
import torch

pytestmark = pytest.mark.gpu


def _P():
    import paper_2212_04180_amd as P
    return P


def _cases():
    P = _P()
    base = dict(sigma=0.1, lr=0.03, init_lo=-2.0, init_hi=2.0, flags=P.FLAG_KEEP_GRAD)
    return [
        ("percall", P.ESConfig(num_dims=300, popsize=64, num_runs=2, seed=1, problem=P.PROB_ROSENBROCK, **base), 20),
        ("fused", P.ESConfig(num_dims=100, popsize=64, num_runs=16, seed=2, problem=P.PROB_RASTRIGIN, **base), 50),
        ("grid", P.ESConfig(num_dims=1000, popsize=128, num_runs=1, seed=3, problem=P.PROB_ROSENBROCK,
                            plan_run_path=3, **base), 30),
        ("percall_big", P.ESConfig(num_dims=20000, popsize=256, num_runs=1, seed=4,
                                   problem=P.PROB_SHIFTED_SPHERE, **base), 8),
    ]


def _run(kind, cfg, T, stream):
    P = _P()
    with torch.cuda.stream(stream):
        es = P.ES(cfg, stream=stream)
        if kind.startswith("percall"):
            fit = torch.empty(cfg.num_runs, cfg.popsize, device="cuda")
            for _ in range(T):
                es.step(fit)
            log = fit
        else:
            log = es.run(T)
        st = es.get_state()
        bx, bf = es.best()
        out = [log, st["m"], st["m1"], st["v"], es.grad(), bx, bf]
        stream.synchronize()
        es.sync()
        out = [x.cpu().numpy() for x in out]
        es.close()
    return out


def test_handles_on_threads_equal_each_run_alone():
    cases = _cases()
    alone = [_run(k, c, T, torch.cuda.Stream()) for k, c, T in cases]
    for rep in range(2):
        results, errors = [None] * len(cases), []

        def work(i):
            try:
                k, c, T = cases[i]
                results[i] = _run(k, c, T, torch.cuda.Stream())
            except Exception as ex:  # reported below, in the main thread
                errors.append((i, repr(ex)))

        threads = [threading.Thread(target=work, args=(i,)) for i in range(len(cases))]
        for th in threads:
            th.start()
        for th in threads:
            th.join(timeout=120)
        assert not any(th.is_alive() for th in threads)
        assert not errors, errors
        for (k, _, _), a, b in zip(cases, alone, results):
            for j, (x, y) in enumerate(zip(a, b)):
                assert x.tobytes() == y.tobytes(), (rep, k, j)
    print(f"{len(cases)} handles on their own threads: the bits of each run alone", flush=True)


def test_init_error_stays_with_its_thread():
    from paper_2212_04180_amd import esmi
    L = esmi.lib()
    msgs = {}
    barrier = threading.Barrier(2)

    def bad():
        cfg = esmi.ESConfig(num_dims=8, popsize=3).cstruct()  # odd population: refused
        h = ctypes.c_void_p()
        barrier.wait()
        rc = L.es_init(ctypes.byref(cfg), None, ctypes.byref(h))
        barrier.wait()
        msgs["bad"] = (rc, L.es_last_error(None))

    def good():
        cfg = esmi.ESConfig(num_dims=8, popsize=4).cstruct()
        h = ctypes.c_void_p()
        barrier.wait()
        rc = L.es_init(ctypes.byref(cfg), None, ctypes.byref(h))
        barrier.wait()
        msgs["good"] = (rc, L.es_last_error(None))
        if rc == esmi.ES_OK:
            L.es_destroy(h)

    ts = [threading.Thread(target=f) for f in (bad, good)]
    for th in ts:
        th.start()
    for th in ts:
        th.join(timeout=60)
    assert msgs["bad"][0] == esmi.ES_ERR_ARG and b"popsize" in msgs["bad"][1]
    assert msgs["good"][0] == esmi.ES_OK and b"popsize" not in msgs["good"][1]
