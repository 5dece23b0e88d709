"""The grid loop of es_run (a cooperative launch of several workgroups per
run, two grid barriers per generation) against the per-call kernels (marked
gpu).  The grid loop replays the per-call plans' chunking and summation
order, so every case must give the same bits: per-generation log, mean, Adam
moments, gradient, best-so-far, sigma and lr.  The per-call path itself is
checked against the oracle stage by stage elsewhere.

Covered: the Rosenbrock D=1000, N=256 workload (the library's default path
for it, with its four-lanes-per-block gradient plan), runs longer than one
launch (256 generations), split gradient plans, evaluate chunkings (fewer
and more chunks than the reduce kernel's 16 slices), one workgroup, more
workgroups than pairs, several runs, and seeded random geometries of every
benchmark problem, both shapings, both signs and the schedules; and the
failure path (waits that give up, forced from the host), reported by es_sync."""
import dataclasses

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _P():
    import paper_2212_04180_amd as P
    return P


def _run(cfg, T):
    P = _P()
    es = P.ES(cfg)
    path = es.run_path
    log = es.run(T)
    st = es.get_state()
    bx, bf = es.best()
    g = es.grad()
    torch.cuda.synchronize()
    es.sync()
    out = [t.cpu().numpy() for t in (log, st["m"], st["m1"], st["v"], bx, bf, g)] + list(es.get_hparams())
    t = es.t
    es.close()
    return path, out, t


def _same(cfg, T):
    pg, og, tg = _run(dataclasses.replace(cfg, plan_run_path=3), T)
    pc, oc, tc = _run(dataclasses.replace(cfg, plan_run_path=1), T)
    assert pg == 3 and pc == 1, (pg, pc)
    assert tg == tc == T
    names = ("log", "m", "m1", "v", "best_x", "best_f", "grad", "sigma", "lr")
    for name, a, b in zip(names, og, oc):
        assert a.tobytes() == b.tobytes(), name
    return og


def _rosenbrock(**kw):
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get("rosenbrock_d1000")
    return dataclasses.replace(cfg, flags=_P().FLAG_KEEP_GRAD, **kw)


def test_default_paths_of_the_workloads():
    # (path, whether the loop's gradient reads the normals its evaluate kept)
    from paper_2212_04180_amd import workloads
    P = _P()
    want = {"sphere_d16": (2, True), "rosenbrock_d1000": (3, True), "rastrigin_r1024": (2, True),
            "shifted_sphere_d1m": (1, False)}
    for name, (path, keeps) in want.items():
        cfg, _ = workloads.get(name)
        es = P.ES(cfg)
        assert (es.run_path, es.run_keeps_normals) == (path, keeps), name
        es.close()


def test_rosenbrock_workload_equals_per_call():
    og = _same(_rosenbrock(), 40)
    assert np.all(np.isfinite(og[1]))
    print("Rosenbrock D=1000 N=256: 40 generations, grid loop bit-identical to the per-call kernels", flush=True)


def test_longer_than_one_launch():
    # 300 generations: two launches (256 + 44), the Adam bias corrections of
    # each in its own kernel arguments; schedules on
    _same(_rosenbrock(sigma_decay=0.99, sigma_final=0.01, lr_decay=0.995, lr_final=0.001), 300)


@pytest.mark.parametrize("kw", [
    dict(popsize=512, plan_tell_split=2),          # split gradient (two workgroups' sums added in split order)
    dict(plan_eval_blocks=7),                      # uneven evaluate chunks (the last one short), 36 chunks
    dict(plan_eval_blocks=1),                      # 250 chunks, 16 per reduce slice
    dict(plan_grid_workgroups=1, num_dims=60),     # one workgroup: no exchange partner
    dict(plan_grid_workgroups=8, popsize=64),      # 8 workgroups: two chunk slices each
    dict(num_runs=3),                              # runs on grid.y, barriers and flags per run
    dict(maximize=1, shaping=1),                   # raw keys, maximised
])
def test_plan_variants(kw):
    _same(_rosenbrock(**kw), 12)


@pytest.mark.parametrize("kw", [dict(), dict(num_runs=3, num_dims=300, popsize=64)])
def test_packed_and_unpacked_launches(kw):
    """The default launch places each run's workgroups on one XCD where the
    device holds the larger launch (the workload; three runs on three XCDs,
    so run r's workgroups are those with x = r mod 8); plan_grid_pack -1
    launches one workgroup per participant.  Both give the per-call bits."""
    a = _same(_rosenbrock(**kw), 20)
    b = _same(_rosenbrock(plan_grid_pack=-1, **kw), 20)
    for x, y in zip(a, b):
        assert np.asarray(x).tobytes() == np.asarray(y).tobytes()


def test_fused_loop_without_kept_normals():
    """1024 runs of 600 dims and 16 members: the fused loop, whose four runs per
    CU (about 49 KB each with the normals kept) would not fit 160 KB of LDS, so
    its gradient regenerates them; the same bits as the per-call kernels."""
    P = _P()
    cfg = P.ESConfig(num_dims=600, popsize=16, num_runs=1024, sigma=0.1, lr=0.02, seed=5, init_lo=-3.0,
                     init_hi=3.0, problem=P.PROB_RASTRIGIN, flags=P.FLAG_KEEP_GRAD)
    es = P.ES(cfg)
    assert (es.run_path, es.run_keeps_normals) == (2, False)
    es.close()
    out = {}
    for path in (2, 1):
        es = P.ES(dataclasses.replace(cfg, plan_run_path=path))
        log = es.run(6)
        st = es.get_state()
        bx, bf = es.best()
        torch.cuda.synchronize()
        out[path] = [x.cpu().numpy() for x in (log, st["m"], st["m1"], st["v"], bx, bf, es.grad())]
        es.close()
    for name, a, b in zip(("log", "m", "m1", "v", "best_x", "best_f", "grad"), out[2], out[1]):
        assert a.tobytes() == b.tobytes(), name


def test_rewound_generation_counter():
    """es_set_state moves t back: the next launch's exchange words must not
    take the values an earlier launch left with the same generation."""
    P = _P()
    cfg = _rosenbrock(num_dims=300, popsize=64)
    out = {}
    for path in (3, 1):
        es = P.ES(dataclasses.replace(cfg, plan_run_path=path))
        assert es.run_path == path
        es.run(12)
        st = es.get_state()
        es.set_state(st["m"], st["m1"], st["v"], 5)  # back to t = 5 with the state of t = 12
        log = es.run(10)
        st = es.get_state()
        torch.cuda.synchronize()
        es.sync()
        out[path] = [x.cpu().numpy() for x in (log, st["m"], st["m1"], st["v"], es.grad())]
        es.close()
    for name, a, b in zip(("log", "m", "m1", "v", "grad"), out[3], out[1]):
        assert a.tobytes() == b.tobytes(), name


def test_wait_that_gives_up_is_reported():
    """The failure path, forced from the host: with plan_grid_spin_limit -1
    every wait of the grid loop gives up at once, so each launch ends early
    (its workgroups leave the kernel at their first wait; a second launch of
    the same es_run sees the flag and leaves too), es_sync reports it, and
    es_set_state clears it.  A spin limit of one poll per wait gives the
    same bits as the default wherever every wait succeeds (the limit is no
    part of the arithmetic): not asserted, since a wait may need a second
    poll."""
    P = _P()
    cfg = _rosenbrock(num_dims=300, popsize=64, plan_run_path=3, plan_grid_spin_limit=-1)
    es = P.ES(cfg)
    assert es.run_path == 3
    st = es.get_state()
    for T in (5, 300):  # one launch, then two
        es.run(T)
        with pytest.raises(P.EsError, match="gave up"):
            es.sync()
        es.set_state(st["m"], st["m1"], st["v"], 0)
        es.sync()
    es.close()
    print("grid loop: forced give-up reported by es_sync and cleared by es_set_state", flush=True)


def test_more_workgroups_than_pairs():
    # 13 dims in four one-block chunks: four workgroups of one chunk each (the
    # nine asked for are lowered to the chunk count), three pairs
    P = _P()
    for problem in (P.PROB_RASTRIGIN, P.PROB_ROSENBROCK):
        cfg = P.ESConfig(num_dims=13, popsize=6, num_runs=2, sigma=0.3, lr=0.05, seed=77, init_lo=-2.0,
                         init_hi=2.0, problem=problem, plan_grid_workgroups=9, flags=P.FLAG_KEEP_GRAD)
        _same(cfg, 20)


def _draw(i):
    P = _P()
    rng = np.random.default_rng(3000 + i)
    while True:
        D = int(np.exp(rng.uniform(0.0, np.log(3000.0))))
        N = 2 * int(np.exp(rng.uniform(0.0, np.log(512.0))))
        R = int(rng.integers(1, 4))
        G = int(rng.choice([0, 0, 1, 2, 3, 4, 8, 16]))
        kw = dict(num_dims=D, popsize=N, num_runs=R, sigma=float(rng.uniform(0.05, 0.5)),
                  lr=float(rng.uniform(0.005, 0.05)), seed=int(rng.integers(0, 1 << 40)), init_lo=-2.0,
                  init_hi=2.0, problem=int(rng.integers(P.PROB_SPHERE, P.PROB_RASTRIGIN + 1)),
                  shaping=int(rng.integers(0, 2)), maximize=int(rng.integers(0, 2)), plan_grid_workgroups=G,
                  plan_tell_split=int(rng.choice([0, 0, 0, 2])), flags=P.FLAG_KEEP_GRAD)
        if rng.integers(0, 2):
            kw.update(sigma_decay=0.97, sigma_final=0.05, lr_decay=0.95, lr_final=0.002)
        cfg = P.ESConfig(**kw)
        es = P.ES(dataclasses.replace(cfg, plan_run_path=3))
        ok = es.run_path == 3  # the drawn plan fits the grid loop's LDS
        es.close()
        if ok:
            return cfg


@pytest.mark.parametrize("i", range(24))
def test_random_grid_loop_equals_per_call(i):
    cfg = _draw(i)
    print("case", i, cfg, flush=True)
    _same(cfg, 9)


def _largest(make, ok, lo, hi):
    """A num_dims in [lo, hi] for which ok(handle) holds and ok(num_dims + 1)
    does not (the largest one where the property is monotonic), by
    bisection; lo must satisfy it."""
    P = _P()
    es = P.ES(make(lo))
    assert ok(es), lo
    es.close()
    while lo < hi:
        mid = (lo + hi + 1) // 2
        es = P.ES(make(mid))
        good = ok(es)
        es.close()
        if good:
            lo = mid
        else:
            hi = mid - 1
    return lo


@pytest.mark.parametrize("problem,N", [("rosenbrock", 256), ("rastrigin", 1024), ("sphere", 64)])
def test_grid_loop_at_its_lds_limit(problem, N):
    """The largest dimension the grid loop takes for a population, counted up
    from the first one it takes (few dims give few workgroups, each holding
    more members' slice sums, so small D can be refused too): its LDS, sized
    on the host, near the 144 KB it may use; the same bits as the per-call
    kernels."""
    P = _P()
    prob = {"rosenbrock": P.PROB_ROSENBROCK, "rastrigin": P.PROB_RASTRIGIN, "sphere": P.PROB_SPHERE}[problem]

    def make(D, path=3):
        return P.ESConfig(num_dims=D, popsize=N, num_runs=1, sigma=0.1, lr=0.02, seed=17, init_lo=-2.0,
                          init_hi=2.0, problem=prob, plan_run_path=path, flags=P.FLAG_KEEP_GRAD)

    def grid(es):
        return es.run_path == 3

    start = None
    for D0 in (16, 64, 256, 1000, 4000):
        es = P.ES(make(D0))
        ok = grid(es)
        es.close()
        if ok:
            start = D0
            break
    assert start is not None
    D = _largest(make, grid, start, 1 << 16)
    print(f"{problem} N={N}: the grid loop up to D={D}", flush=True)
    _same(make(D, 0), 4)


def test_fused_loop_at_its_lds_limit():
    """1024 runs of 64 members: the largest dimension the fused loop takes by
    default (its workgroup's LDS at the limit), and the largest for which it
    still keeps the normals; both the same bits as the per-call kernels."""
    P = _P()

    def make(D, path=0):
        return P.ESConfig(num_dims=D, popsize=64, num_runs=1024, sigma=0.2, lr=0.02, seed=23, init_lo=-3.0,
                          init_hi=3.0, problem=P.PROB_RASTRIGIN, plan_run_path=path, flags=P.FLAG_KEEP_GRAD)

    d_fused = _largest(make, lambda es: es.run_path == 2, 8, 1 << 14)
    d_keep = _largest(make, lambda es: es.run_path == 2 and es.run_keeps_normals, 8, d_fused)
    print(f"fused loop up to D={d_fused}, normals kept up to D={d_keep}", flush=True)
    for D in sorted({d_keep, d_fused}):
        out = {}
        for path in (2, 1):
            es = P.ES(make(D, path))
            log = es.run(3)
            st = es.get_state()
            bx, bf = es.best()
            torch.cuda.synchronize()
            out[path] = [x.cpu().numpy() for x in (log, st["m"], st["m1"], st["v"], bx, bf, es.grad())]
            es.close()
        for name, a, b in zip(("log", "m", "m1", "v", "best_x", "best_f", "grad"), out[2], out[1]):
            assert a.tobytes() == b.tobytes(), (D, name)


@pytest.mark.parametrize("problem", ["rosenbrock", "sphere"])
def test_overflowing_fitness_loops_equal_per_call(problem):
    """Means near 1e20: the fitness overflows to inf (and Rosenbrock's terms
    to NaN), so the order keys hold ties and NaN, and both loops must still
    give the per-call bits (log, state, best-so-far)."""
    P = _P()
    prob = {"rosenbrock": P.PROB_ROSENBROCK, "sphere": P.PROB_SPHERE}[problem]
    grid = P.ESConfig(num_dims=300, popsize=64, num_runs=2, sigma=0.1, lr=0.05, seed=31, init_lo=-1e20,
                      init_hi=1e20, problem=prob, flags=P.FLAG_KEEP_GRAD)
    og = _same(grid, 6)
    assert not np.all(np.isfinite(og[0]))  # the log carries the overflow
    fused = dataclasses.replace(grid, num_dims=40, popsize=32, num_runs=200)
    es = P.ES(fused)
    assert es.run_path == 2
    es.close()
    out = {}
    for path in (2, 1):
        es = P.ES(dataclasses.replace(fused, plan_run_path=path))
        log = es.run(6)
        st = es.get_state()
        bx, bf = es.best()
        torch.cuda.synchronize()
        out[path] = [x.cpu().numpy() for x in (log, st["m"], st["m1"], st["v"], bx, bf, es.grad())]
        es.close()
    for name, a, b in zip(("log", "m", "m1", "v", "best_x", "best_f", "grad"), out[2], out[1]):
        assert a.tobytes() == b.tobytes(), name
