"""Throughput of one batched OpenAI-ES generation (ask + evaluate + tell) on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
                [--no-other-workloads]

A step is one whole generation of the per-call path (es_ask, es_eval,
es_tell) on the synthetic workload (default: shifted sphere, D = 1e6,
N = 2048, R = 1).  With the default workload the same run also times the
other four workloads (the neuroevolution MLP through the per-call path; the
sphere D = 16, Rosenbrock D = 1000 and R = 1024 Rastrigin runs through
es_run) under "other_workloads".  Prints ONE JSON line on stdout;
diagnostics go to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X public figures: 256 CUs at 2.4 GHz; fp32 vector 157.3 TFLOP/s, i.e.
# 7.86e13 full-rate VALU lane-ops/s (an FMA counts two flops); HBM3E 8 TB/s.
VALU_PEAK = 157.3e12 / 2.0  # lane-op slots/s
HBM_PEAK = 8.0e12
BF16_MFMA_PEAK = 2.5e15  # dense bf16 matrix FLOP/s
# Neuroevolution MLP 64-256-256-16 on 256 inputs: 2 flops per weight per input
MLP_FLOPS_PER_MEMBER = 2 * 256 * (64 * 256 + 256 * 256 + 256 * 16)

# Algorithmic VALU work, in full-rate lane-op slots per Philox block of one
# antithetic pair (4 dims x 2 members).  Issue costs measured on gfx950
# relative to v_fma_f32 (1): v_mad_u64_u32, v_mul_hi/lo_u32, v_cvt_*, fp64
# fma/add 2; v_log/v_sqrt/v_sin/v_cos 4; bitwise, shifts, fp32 add/mul/fma 1.
#   Philox-4x32-10: 20 x 32x32->64 product (2) + 20 x three-input xor (1)      = 60
#   Box-Muller: 4 shift + 4 cvt (2) + 4 x 2^-24 scale (the radius words'
#     +1 folded into their scale as one fma) + 2 log2 (4) + 2 x (-2 ln 2)
#     + 2 sqrt (4) + 2 sin (4) + 2 cos (4) + 4 (r * trig)                      = 54
#   members (both signs): 8 fma for x plus the problem's terms, and the fold
#     of each member's fp32 block sum into fp64 (2 x (cvt 2 + add 2) = 8):
#     sphere 8 squares -> 24; shifted sphere 8 sub + 8 squares -> 32;
#     Rosenbrock 6 ops x 4 terms x 2 -> 64; Rastrigin 8 ops x 8 -> 80 (fract of
#     |x| (1), cos (4), -a cos (1), x^2 + that (1), the add (1)).
PHILOX_BM = 60 + 54
EVAL_SLOTS_PER_PAIR_BLOCK = {"sphere": PHILOX_BM + 24, "shifted_sphere": PHILOX_BM + 32,
                             "rosenbrock": PHILOX_BM + 64, "rastrigin": PHILOX_BM + 80}
# tell: Philox + Box-Muller + 4 fma (w * eps) + the fp64 fold every 16 pairs
TELL_SLOTS_PER_PAIR_BLOCK = PHILOX_BM + 4 + 1
# es_run's code paths (es_run_path); where a loop's gradient reads the
# normals its evaluate kept in LDS (es_run_path's keeps_normals), its work per
# pair-block omits one Philox block and Box-Muller
RUN_PATHS = {1: "per-call kernels", 2: "fused loop (k_run_fused, one workgroup per run)",
             3: "grid loop (k_run_grid, a cooperative launch of several workgroups per run)"}
# per-dimension sigma (PGPE, SNES): evaluate moves each dim's sigma into a
# VGPR (4 movs per block); tell adds the second sum, 4 fma (z*z - 1) + 4 fma
EVAL_VEC_EXTRA = 4
TELL_TWO_EXTRA = 8


def kernel_source_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in ("es_device.hpp", "es_kernels.hip"):
        with open(os.path.join(ROOT, "paper_2212_04180_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def profiled_traffic(workload, key="eval_hbm_bytes_request_sized", cast=int):
    """A figure of the evaluate kernel from the committed rocprofv3 counter
    summary of this workload, or None if there is none or the kernel sources
    changed since the counters were taken.  The default key is the HBM bytes
    per launch with each read request priced at its size (the evaluate
    kernel's scalar-cache reads are 64-B requests, the copy's 128-B);
    eval_hbm_bytes_per_launch is the copy-calibrated FETCH_SIZE + WRITE_SIZE,
    eval_valu_instructions_per_pair_block the VALU instructions the kernel
    issues per pair-block (SQ_INSTS_VALU per wave of 64 pairs)."""
    path = os.path.join(ROOT, "profiles", f"k_eval_bbob_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_sha256():
        return None
    try:
        return cast(kv[key])
    except (KeyError, ValueError):
        return None


def issue_profile(key):
    """A figure of the committed issue-rate summary (valu_issue_costs_gfx950.txt),
    or None if it is missing or the probe source changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "valu_issue_costs_gfx950.txt")
    src = os.path.join(ROOT, "paper_2212_04180_amd", "csrc", "es_probe.hip")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip().split()[0] if v.strip() else ""
    with open(src, "rb") as fh:
        if kv.get("probe_source_sha256") != hashlib.sha256(fh.read()).hexdigest():
            return None
    try:
        return float(kv[key])
    except (KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="shifted_sphere_d1m")
    ap.add_argument("--path", choices=["percall", "run"], default="percall",
                    help="percall: es_ask/es_eval/es_tell per generation; run: es_run over all K generations")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="time only --workload (the default workload also times the other four)")
    ap.add_argument("--cpu-sample-dims", type=int, default=0)
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this size (HBM counter calibration)")
    ap.add_argument("--issue-costs", action="store_true",
                    help="measure the issue cost of the instructions behind the slot weights (libesmi_probe.so) "
                         "and print that JSON line instead")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(cfg, sample_dims):
    """The oracle as it stands, on the host cores, on a bounded sample of the
    workload: one whole generation of the same strategy restricted to its
    first `sample_dims` dims (same N, R, problem), once on one thread and
    once on all the threads OpenMP is given (the oracle's parallel loops give
    the same bits).  Scaled to member-dims/s; the all-threads figure is the
    value, `cores` the threads it used, `host_cores` the cores this process
    may run on."""
    from oracle import oracle as O
    legs = {}
    for threads in (1, 0):
        O.set_threads(threads)
        used = O.get_threads()
        legs[threads] = (used, _oracle_generation(O, cfg, sample_dims))
    O.set_threads(0)
    md = cfg.num_runs * cfg.popsize * sample_dims
    (n1, dt1), (nt, dtn) = legs[1], legs[0]
    return {"value": md / dtn, "unit": "member-dims/s", "cores": nt, "kind": "oracle",
            "host_cores": len(os.sched_getaffinity(0)),
            "single_thread": {"value": md / dt1, "seconds": dt1},
            "sample": f"1 generation (ask+eval+tell) of the same workload on its first {sample_dims} dims "
                      f"(R={cfg.num_runs}, N={cfg.popsize}): {dtn:.2f} s on {nt} threads, "
                      f"{dt1:.2f} s on one"}


def _oracle_generation(O, cfg, sample_dims):
    oc = O.OracleConfig(num_dims=sample_dims, popsize=cfg.popsize, num_runs=cfg.num_runs, sigma=cfg.sigma,
                        lr=cfg.lr, beta1=cfg.beta1, beta2=cfg.beta2, eps=cfg.eps, maximize=cfg.maximize,
                        shaping=cfg.shaping, seed=cfg.seed, init=cfg.init, init_lo=cfg.init_lo,
                        init_hi=cfg.init_hi, problem=cfg.problem, rastrigin_a=cfg.rastrigin_a,
                        mlp_batch=cfg.mlp_batch, mlp_bf16=cfg.mlp_bf16, mlp_tanh_out=cfg.mlp_tanh_out,
                        sigma_decay=cfg.sigma_decay, sigma_final=cfg.sigma_final, lr_decay=cfg.lr_decay,
                        lr_final=cfg.lr_final, w_decay=cfg.w_decay, strategy=cfg.strategy,
                        optimizer=cfg.optimizer, sigma_lr=cfg.sigma_lr, sigma_max_change=cfg.sigma_max_change,
                        clipup_max_speed=cfg.clipup_max_speed, clipup_momentum=cfg.clipup_momentum,
                        snes_temperature=cfg.snes_temperature, elite_ratio=cfg.elite_ratio)
    es = O.OracleES(oc)
    t0 = time.perf_counter()
    es.step()
    return time.perf_counter() - t0


def time_workload(P, torch, name, K, W, path, dev, stream, copy_mib=0):
    """Times K generations of workload `name` (after W warm-up generations)
    through the per-call path or es_run; returns the timings and roofline."""
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get(name)
    es = P.ES(cfg, device=dev, stream=stream)
    run_path = es.run_path if path == "run" else 1
    keeps = path == "run" and es.run_keeps_normals
    R, N, D = cfg.num_runs, cfg.popsize, cfg.num_dims
    fit = torch.empty(R, N, device=dev)
    if copy_mib:
        n = copy_mib * (1 << 20) // 4
        src = torch.ones(n, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copy calibration: {n * 4} bytes read + {n * 4} bytes written")
        del src, dst

    if path == "run":
        es.run(W, log=False)
    else:
        for _ in range(W):
            es.step(fit)
    torch.cuda.synchronize()

    # Two HIP events per generation time the dominant kernel, the main
    # evaluate kernel: es_eval_timed has its dispatch record them
    # (hipExtLaunchKernel), so the timed stream holds no marker packets (an
    # event record between kernels leaves the stream idle for a few
    # microseconds).  The rest of the generation (fitness reduce, ranks,
    # gradient, update) runs from one generation's stop event to the next
    # one's start event.  Each event is recorded once here, outside the timed
    # region, so that it exists.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    for pair in ev:
        for e in pair:
            e.record(stream)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    if path == "run":
        es.run(K, log=False)
    else:
        for k in range(K):
            es.ask()
            es.eval(fit, events=ev[k])
            es.tell(fit)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    # a grid-loop launch whose waits gave up ends early: raise rather than
    # report its short time
    es.sync()
    ms = start.elapsed_time(end) / K
    if path == "run":
        eval_ms = rest_ms = None  # es_run has no phase boundaries to time
    else:
        eval_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / K
        rest_ms = sum(ev[k][1].elapsed_time(ev[k + 1][0] if k + 1 < K else end) for k in range(K)) / K
    es.close()
    value = R * N * D / (ms * 1e-3)
    phases = f" (eval kernel {eval_ms:.4f}, rest {rest_ms:.4f})" if eval_ms is not None else ""
    log(f"[bench] {name} ({path}, {RUN_PATHS[run_path]}): {ms:.4f} ms/gen{phases}, wall {wall:.3f}s for {K} gens, "
        f"{value:.4e} member-dims/s")

    prob = {P.PROB_SHIFTED_SPHERE: "shifted_sphere", P.PROB_SPHERE: "sphere", P.PROB_RASTRIGIN: "rastrigin",
            P.PROB_ROSENBROCK: "rosenbrock"}.get(cfg.problem)
    pair_blocks = R * (N // 2) * ((D + 3) // 4)
    roof = None
    if prob is not None and path == "percall":
        vec = cfg.strategy != P.STRAT_OPENAI_ES
        eval_slots = EVAL_SLOTS_PER_PAIR_BLOCK[prob] + (EVAL_VEC_EXTRA if vec else 0)
        tell_slots = TELL_SLOTS_PER_PAIR_BLOCK + (TELL_TWO_EXTRA if vec else 0)
        tell_items = pair_blocks
        if cfg.strategy == P.STRAT_SEP_CMA:
            # independent members: a second Philox block and Box-Muller per
            # pair-block; the gradient sums run over the mu elites
            eval_slots += PHILOX_BM
            mu = max(1, int(cfg.elite_ratio * N))
            tell_items = R * mu * ((D + 3) // 4)
        achieved = pair_blocks * eval_slots / (eval_ms * 1e-3)
        tell_achieved = tell_items * tell_slots / (rest_ms * 1e-3)
        issued = profiled_traffic(name, "eval_valu_instructions_per_pair_block", float)
        best_stream = issue_profile("fma_f32_vvv_frac_of_slot_peak")
        roof = {"bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK / 1e12,
                "unit": "T VALU lane-op slots/s", "frac": achieved / VALU_PEAK,
                "traffic": profiled_traffic(name),
                "traffic_copy_scaled": profiled_traffic(name, "eval_hbm_bytes_per_launch"),
                "kernel": "k_eval_bbob (fused sample+evaluate)",
                "kernel_ms": eval_ms, "slots_per_pair_block": eval_slots,
                "pair_blocks_per_launch": pair_blocks,
                "issued_instructions_per_pair_block": issued,
                "issued_frac": None if issued is None else pair_blocks * issued / (eval_ms * 1e-3) / VALU_PEAK,
                "best_single_instruction_stream_frac": best_stream,
                "tell": {"kernel": "k_eval_reduce + k_rank + k_tell (+ the strategy's update passes): the rest "
                                   "of the generation", "kernel_ms": rest_ms, "achieved": tell_achieved / 1e12,
                         "frac": tell_achieved / VALU_PEAK, "slots_per_pair_block": tell_slots}}
    if prob is not None and path == "run" and cfg.strategy == P.STRAT_OPENAI_ES:
        # whole generations: evaluate and gradient slots over the timed launch(es)
        slots = EVAL_SLOTS_PER_PAIR_BLOCK[prob] + TELL_SLOTS_PER_PAIR_BLOCK - (PHILOX_BM if keeps else 0)
        achieved = pair_blocks * slots / (ms * 1e-3)
        roof = {"bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK / 1e12,
                "unit": "T VALU lane-op slots/s", "frac": achieved / VALU_PEAK, "traffic": None,
                "kernel": "es_run: " + RUN_PATHS[run_path], "keeps_normals": bool(keeps),
                "kernel_ms": ms, "slots_per_pair_block": slots, "pair_blocks_per_generation": pair_blocks}
    if cfg.problem == P.PROB_MLP and path == "percall":
        flops = R * N * MLP_FLOPS_PER_MEMBER
        achieved = flops / (eval_ms * 1e-3)
        tell_achieved = pair_blocks * TELL_SLOTS_PER_PAIR_BLOCK / (rest_ms * 1e-3)
        roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": BF16_MFMA_PEAK / 1e12, "unit": "TFLOP/s",
                "frac": achieved / BF16_MFMA_PEAK, "traffic": None,
                "kernel": "k_eval_mlp (the bf16 MFMA forward of every member)",
                "kernel_ms": eval_ms, "flops_per_launch": flops,
                "generation_frac": flops / (ms * 1e-3) / BF16_MFMA_PEAK,
                "tell": {"kernel": "k_rank + k_tell (with the next generation's teacher rows) + k_tell_fold: "
                                   "the rest of the generation", "kernel_ms": rest_ms,
                         "achieved": tell_achieved / 1e12, "unit": "T VALU lane-op slots/s",
                         "frac": tell_achieved / VALU_PEAK}}
    return {"cfg": cfg, "prob": prob, "ms": ms, "eval_ms": eval_ms, "rest_ms": rest_ms, "value": value,
            "roofline": roof, "K": K, "run_path": RUN_PATHS[run_path]}


# Instructions of the probe (include/esmi_probe.h) in its enum order, the
# launch's loop count for each (a few milliseconds per launch), and the slot
# weight the algorithmic counts above give each.
PROBE_OPS = [("v_fma_f32", 20000, 1), ("v_bitop3_b32", 20000, 1), ("v_mad_u64_u32", 10000, 2),
             ("v_cvt_f32_u32", 20000, 2), ("v_cvt_pk_bf16_f32", 20000, None), ("v_log_f32", 5000, 4),
             ("v_exp_f32", 5000, None), ("v_rcp_f32", 5000, None), ("v_sqrt_f32", 5000, 4), ("v_sin_f32", 5000, 4),
             ("v_cos_f32", 5000, 4), ("v_fma_f64", 10000, 2), ("v_add_f64", 10000, 2),
             ("v_mfma_f32_16x16x32_bf16", 2000, None), ("v_mul_f32", 20000, 1), ("v_xor_b32", 20000, 1),
             ("v_fma_f32 (three VGPR sources)", 20000, 1)]


def issue_costs(torch, dev, stream):
    """Issue rate of each probed instruction on all 256 CUs (eight waves per
    SIMD, eight independent chains per lane), timed with HIP events; the
    slots of an instruction are v_fma_f32's rate over its rate."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2212_04180_amd", "libesmi_probe.so"))
    lib.es_probe_issue.restype = ctypes.c_int32
    lib.es_probe_issue.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    lib.es_probe_threads.restype = ctypes.c_int64
    lib.es_probe_chains.restype = ctypes.c_int32
    threads, chains = lib.es_probe_threads(), lib.es_probe_chains()
    sink = torch.empty(threads, dtype=torch.int32, device=dev)
    out = {}
    for op, (name, iters, model) in enumerate(PROBE_OPS):
        times = []
        for rep in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            rc = lib.es_probe_issue(op, iters, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
            e1.record(stream)
            if rc != 0:
                raise RuntimeError(f"probe {name}: hip error {rc}")
            torch.cuda.synchronize()
            if rep:
                times.append(e0.elapsed_time(e1) * 1e-3)
        t = min(times)
        wave_instr = threads // 64 * iters * chains
        out[name] = {"seconds": t, "wave_instructions": wave_instr, "lane_ops_per_s": wave_instr * 64 / t,
                     "model_slots": model}
    fma = out["v_fma_f32"]["lane_ops_per_s"]
    for name, v in out.items():
        v["slots"] = fma / v["lane_ops_per_s"]
        if name.startswith("v_mfma"):
            v["flops_per_s"] = v["wave_instructions"] * 16384 / v["seconds"]
            v["frac_of_bf16_peak"] = v["flops_per_s"] / BF16_MFMA_PEAK
    return {"fma_f32_lane_ops_per_s": fma, "frac_of_slot_peak": fma / VALU_PEAK, "instructions": out}


# The other workloads the default run also times: name -> (path, generations
# timed, warm-up generations).  The per-call path for the MLP (its roofline
# is the evaluate kernel's share of the bf16 MFMA peak), es_run for the three
# small ones (their configured generation counts, one es_run call each).
OTHER_WORKLOADS = {"mlp_teacher": ("percall", 20, 3), "sphere_d16": ("run", 100, 100),
                   "rosenbrock_d1000": ("run", 500, 50), "rastrigin_r1024": ("run", 200, 20)}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library runs every strategy on a single MI355X and "
              "sharding over several GPUs is not implemented", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2212_04180_amd as P

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    if args.issue_costs:
        ic = issue_costs(torch, dev, stream)
        for name, v in ic["instructions"].items():
            log(f"[issue] {name:26s} {v['lane_ops_per_s']:.3e} lane-ops/s  {v['slots']:.2f} slots"
                + (f" (model {v['model_slots']})" if v["model_slots"] is not None else ""))
        print(json.dumps({"issue_costs": ic}), flush=True)
        return
    res = time_workload(P, torch, args.workload, args.steps, args.warmup, args.path, dev, stream,
                        args.copy_calibration_mib)
    cfg, prob, ms, value = res["cfg"], res["prob"], res["ms"], res["value"]
    R, N, D = cfg.num_runs, cfg.popsize, cfg.num_dims

    others = None
    if args.workload == "shifted_sphere_d1m" and not args.no_other_workloads:
        others = {}
        for name, (path, K, W) in OTHER_WORKLOADS.items():
            o = time_workload(P, torch, name, K, W, path, dev, stream)
            oc = o["cfg"]
            others[name] = {"path": path, "code_path": o["run_path"], "steps": K, "ms_per_step": o["ms"],
                            "generations_per_s": 1e3 / o["ms"],
                            "value": o["value"], "unit": "member-dims/s",
                            "num_runs": oc.num_runs, "popsize": oc.popsize, "num_dims": oc.num_dims,
                            "eval_kernel_ms": o["eval_ms"], "rest_ms": o["rest_ms"], "roofline": o["roofline"]}

    # HBM reading of the metric: the same generation with the noise stored
    # (written once by evaluate, read once by tell) moves 4 B per member-dim.
    # An equivalence, not a share of HBM bandwidth: the path stores no noise.
    hbm_equiv = {"bytes_per_member_dim": 4.0, "peak_member_dims_per_s": HBM_PEAK / 4.0,
                 "equivalent_frac": value / (HBM_PEAK / 4.0),
                 "reading": "throughput of a noise-storing design at the full 8 TB/s; not a share of HBM "
                            "bandwidth (this path regenerates the noise and moves about 50 MB per generation)"}

    cpu = None
    if not args.no_cpu_baseline:
        sd = args.cpu_sample_dims or max(4, min(D, int(4.0e8 // (R * N))))
        cpu = cpu_baseline(cfg, sd)
        log(f"[bench] oracle sample: {cpu['sample']} -> {cpu['value']:.3e} member-dims/s "
            f"({cpu['cores']} threads; host cores {cpu['host_cores']})")

    out = {
        "metric": "member-dims/sec per ES generation (ask+eval+tell)",
        "value": value,
        "unit": "member-dims/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.problem == P.PROB_MLP else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "path": args.path, "num_runs": R, "popsize": N, "num_dims": D,
                   "problem": prob or "mlp", "sigma": cfg.sigma, "lr": cfg.lr,
                   "strategy": {0: "openai_es", 1: "pgpe", 2: "snes", 3: "sep_cma_es"}[cfg.strategy],
                   "optimizer": "clipup" if cfg.optimizer == P.OPT_CLIPUP and cfg.strategy != P.STRAT_SNES else
                   ({0: "adam", 1: "adam", 2: "snes natural gradient", 3: "cma recombination"}[cfg.strategy]),
                   "generations_per_s": 1e3 / ms, "eval_kernel_ms": res["eval_ms"], "rest_ms": res["rest_ms"]},
        "roofline": res["roofline"],
        "hbm_equivalent": hbm_equiv,
        "cpu_baseline": cpu,
        "other_workloads": others,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
