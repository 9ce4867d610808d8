"""Build the gfx950 shared library ``libhptt.so`` in-tree with hipcc.

``python -m paper_1704_04374_amd.build`` compiles every source under ``csrc/``
(HIP kernels and the host half of the C ABI) into
``paper_1704_04374_amd/libhptt.so``.  Objects go to ``_build/`` at the
repository root.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libhptt.so")
# Contractions (transposition - GEMM - transposition) link rocBLAS, so they
# live in a library of their own on top of libhptt.so.
CONTRACT_LIB = os.path.join(PKG, "libhptt_contract.so")
CONTRACT_SOURCES = ["contract.hip"]

ARCH = "gfx950"
# the tile kernel instantiations are split over six files so they compile in parallel
SOURCES = ["tile_f32_fast.hip", "tile_f32_shifted.hip", "tile_f32_general.hip", "tile_shared.hip",
           "tile_direct.hip", "tile_f64.hip", "kernels.hip",
           "yardstick.hip", "api.cpp", "plan.cpp", "autotune.cpp"]

# -ffp-contract=off: alpha*a + beta*b is two roundings and an add, never an
# FMA.  The packed-fp32 feature is switched off for every HIP file.
COMMON = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Wall",
          f"-I{INCLUDE}", f"-I{CSRC}"]
HIP_ONLY = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang",
            "-packed-fp32-ops"]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return path


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [hipcc(), *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip", *HIP_ONLY]
    else:  # host code only: no device pass
        cmd[1:1] = ["-x", "hip", f"--offload-arch={ARCH}", "--offload-host-only"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile all sources and link ``libhptt.so``; return its path."""
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking libhptt.so failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    with cf.ThreadPoolExecutor(max_workers=len(CONTRACT_SOURCES)) as ex:
        cobjs = list(ex.map(_compile, CONTRACT_SOURCES))
    tmp = CONTRACT_LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *cobjs, "-o", tmp, f"-L{PKG}",
           "-lhptt", "-lrocblas", "-Wl,-rpath,$ORIGIN"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking libhptt_contract.so failed:\n{' '.join(cmd)}\n"
                           f"{r.stdout}{r.stderr}")
    os.replace(tmp, CONTRACT_LIB)
    if verbose:
        print(f"built {LIB} and {CONTRACT_LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
