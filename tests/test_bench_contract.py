"""bench.py pieces that run without a GPU: the oracle baseline on a small
sample of every benchmark workload, and the refusal of more than one GPU."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


@pytest.mark.parametrize("name", ["sphere_d16", "rosenbrock_d1000", "rastrigin_r1024", "shifted_sphere_d1m",
                                  "pgpe_shifted_sphere_d1m", "snes_shifted_sphere_d1m", "sepcma_shifted_sphere_d1m",
                                  "clipup_shifted_sphere_d1m"])
def test_cpu_baseline_runs_the_oracle_on_a_sample(name):
    sys.path.insert(0, ROOT)
    import bench
    from paper_2212_04180_amd import workloads
    cfg, _ = workloads.get(name)
    if cfg.num_runs > 8:
        cfg.num_runs = 8  # keep the CPU test short
    out = bench.cpu_baseline(cfg, 8)
    assert out["kind"] == "oracle" and out["unit"] == "member-dims/s"
    assert out["cores"] >= 1 and out["host_cores"] == len(os.sched_getaffinity(0))
    assert out["value"] > 0 and out["single_thread"]["value"] > 0 and "8 dims" in out["sample"]
    from oracle import oracle as O
    assert O.get_threads() == out["cores"]  # the default restored after the one-thread leg


def test_other_workloads_are_the_remaining_four():
    sys.path.insert(0, ROOT)
    import bench
    from paper_2212_04180_amd import workloads
    assert set(bench.OTHER_WORKLOADS) == {"mlp_teacher", "sphere_d16", "rosenbrock_d1000", "rastrigin_r1024"}
    for name, (path, K, W) in bench.OTHER_WORKLOADS.items():
        workloads.get(name)
        assert path in ("percall", "run") and K > 0 and W >= 0
