"""The C-ABI library loads and exports every symbol include/esmi.h declares
(CPU only: no compute call is made)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "esmi.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return re.findall(r"\b(es_[a-z_]+)\s*\(", src)


def test_header_declares_the_boundary():
    names = _declared()
    for must in ("es_init", "es_ask", "es_eval", "es_tell", "es_run", "es_destroy"):
        assert must in names


def test_library_exports_every_declared_symbol():
    from paper_2212_04180_amd import esmi
    L = esmi.lib()
    names = _declared()
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing
    assert sorted(set(names)) == sorted(set(esmi.EXPORTS))


def test_status_strings_and_init_error_without_gpu_work():
    from paper_2212_04180_amd import esmi
    L = esmi.lib()
    assert L.es_status_string(0) == b"ok"
    assert L.es_run_path(None, None) == 0 and L.es_generation(None) == -1
    assert L.es_status_string(-2).startswith(b"call out of")
    # an invalid config is rejected before any device call
    cfg = esmi.ESConfig(num_dims=8, popsize=3).cstruct()
    h = ctypes.c_void_p()
    assert L.es_init(ctypes.byref(cfg), None, ctypes.byref(h)) == esmi.ES_ERR_ARG
    assert b"popsize" in L.es_last_error(None)


def test_config_struct_has_no_padding():
    # no padding bytes: checkpoints compare the config byte for byte
    from paper_2212_04180_amd import esmi
    fields = sum(ctypes.sizeof(t) for _, t in esmi._Config._fields_)
    assert ctypes.sizeof(esmi._Config) == fields == 168


def test_product_does_not_reach_the_oracle():
    pkg = os.path.join(ROOT, "paper_2212_04180_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".hpp", ".h")):
                text = open(os.path.join(dirpath, fn)).read()
                assert "oracle" not in text.lower().replace("the oracle", ""), fn


def test_probe_library_exports_its_header():
    """The issue-rate probe (a measurement aid of the benchmark) is a library
    of its own: the generation's library does not carry it."""
    src = open(os.path.join(ROOT, "include", "esmi_probe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(es_probe_[a-z_]+)\s*\(", src)
    assert set(names) == {"es_probe_issue", "es_probe_threads", "es_probe_chains"}
    L = ctypes.CDLL(os.path.join(ROOT, "paper_2212_04180_amd", "libesmi_probe.so"))
    for n in names:
        assert hasattr(L, n)
    L.es_probe_threads.restype = ctypes.c_int64
    assert L.es_probe_threads() == 2048 * 256
    from paper_2212_04180_amd import esmi
    assert not hasattr(esmi.lib(), "es_probe_issue")


def test_population_limits_are_validated_without_gpu_work():
    """Up to 16384 members the ranks are counted in LDS; beyond, the sort-based
    ranks take over, up to 2^24 members; launch-plan fields in range
    (rejected before any device call)."""
    from paper_2212_04180_amd import esmi
    L = esmi.lib()
    h = ctypes.c_void_p()
    for kw, msg in ((dict(popsize=(1 << 24) + 2), b"2^24"),
                    (dict(popsize=16386, plan_rank_path=1), b"plan_rank_path 1"),
                    (dict(popsize=64, plan_rank_path=3), b"plan_rank_path must be"),
                    (dict(popsize=(1 << 20), num_runs=4096), b"2^31"),
                    (dict(popsize=64, plan_run_path=4), b"plan_run_path must be"),
                    (dict(popsize=64, plan_grid_workgroups=17), b"plan_grid_workgroups"),
                    (dict(popsize=64, plan_grid_workgroups=-1), b"plan_grid_workgroups"),
                    (dict(popsize=64, plan_grid_spin_limit=-2), b"plan_grid_spin_limit"),
                    (dict(popsize=64, plan_grid_pack=1), b"plan_grid_pack"),
                    (dict(popsize=64, plan_grid_pack=-2), b"plan_grid_pack")):
        cfg = esmi.ESConfig(num_dims=8, **kw).cstruct()
        assert L.es_init(ctypes.byref(cfg), None, ctypes.byref(h)) == esmi.ES_ERR_ARG, kw
        assert msg in L.es_last_error(None), (kw, L.es_last_error(None))
