"""Build step of the HIP library: compiles csrc/ into libesmi.so for gfx950.

Called by ``__graft_entry__.build()`` and usable by hand (``python -m
paper_2212_04180_amd.build``).  Always recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libesmi.so")
SOURCES = ["es_kernels.hip", "es_mlp.hip", "es_rank_sort.hip", "es_api.cpp"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def compile_flags():
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra",
        "-Wno-unused-parameter",
        # no packed fp32 math: keep v_pk_{add,mul,fma}_f32 out of the code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
    ]


PROBE_SRC = "es_probe.hip"
PROBE_LIB = os.path.join(PKG, "libesmi_probe.so")


def build_probe(cc: str, verbose: bool = False) -> str:
    """The issue-rate probe behind the benchmark's slot weights (a separate
    library; the generation never loads it)."""
    tmp = PROBE_LIB + ".tmp%d" % os.getpid()
    cmd = [cc, *compile_flags(), "-shared", "-x", "hip", os.path.join(CSRC, PROBE_SRC), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True, stderr=None if verbose else subprocess.PIPE)
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


def build(verbose: bool = False) -> str:
    cc = hipcc()
    build_probe(cc, verbose)
    objs = []
    for src in SOURCES:
        obj = os.path.join(CSRC, src + ".o")
        cmd = [cc, *compile_flags(), "-c", "-x", "hip", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True, stderr=None if verbose else subprocess.PIPE)
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    for o in objs:
        os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
