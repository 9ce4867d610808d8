"""Build the test-only host emulator library ``libhptt_emulate.so``.

It compiles ``emulate.cpp`` (host code that runs the kernels' phase functions
with checked memory) together with the library's plan builder and host ABI,
for the host only.  The product library ``libhptt.so`` never contains it.
"""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_1704_04374_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libhptt_emulate.so")


def build() -> str:
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    srcs = [os.path.join(HERE, "emulate.cpp"), os.path.join(CSRC, "plan.cpp"),
            os.path.join(CSRC, "api.cpp")]
    tmp = f"{LIB}.tmp{os.getpid()}"  # one per process: test workers may build at once
    cmd = [hipcc, "-x", "hip", "--offload-host-only", "-O2", "-g", "-std=c++17", "-fPIC",
           "-shared", "-ffp-contract=off", "-Wall", f"-I{INCLUDE}", f"-I{CSRC}", *srcs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building the emulator failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
