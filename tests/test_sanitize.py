"""The host code built with AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): the plan builder, the autotuner's candidate enumeration, the
kernels' phase functions under the host emulator and the CPU oracle, driven
by tests/sanitize/host_check.cpp over random, sub-tensor, high-rank and
misaligned problems (each compared bit for bit with the oracle) and strided
dry runs of the named full-size workloads.  Any sanitizer report aborts the
program, so the test passes only on a clean run."""
from __future__ import annotations

import concurrent.futures
import os
import subprocess

import pytest

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)
CSRC = os.path.join(ROOT, "paper_1704_04374_amd", "csrc")
BUILD = os.path.join(ROOT, "_build", "sanitize")
CLANG = "/opt/rocm/lib/llvm/bin/clang"


def _compile(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}{r.stderr}"


def _stale(out: str, src: str) -> bool:
    """True when `out` is missing or older than `src` or any header it may include."""
    if not os.path.exists(out):
        return True
    deps = [src] + [os.path.join(d, f) for d in (CSRC, os.path.join(ROOT, "include"))
                    for f in os.listdir(d) if f.endswith(".h")]
    return any(os.path.getmtime(x) > os.path.getmtime(out) for x in deps)


def _build() -> str:
    if not os.path.exists(CLANG):
        pytest.skip("ROCm clang not found")
    os.makedirs(BUILD, exist_ok=True)
    # host code only: -Xarch_host applies each sanitizer flag to the host pass
    san = ["-Xarch_host", "-fsanitize=address,undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g1", "-O0"]
    oracle_src = os.path.join(ROOT, "oracle", "oracle.c")
    jobs = [(oracle_src, [CLANG, "-x", "c", "-std=c99", "-ffp-contract=off", *san])]
    for src in (os.path.join(TESTS, "sanitize", "host_check.cpp"),
                os.path.join(TESTS, "emulator", "emulate.cpp"),
                os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "api.cpp"),
                os.path.join(CSRC, "autotune.cpp")):
        jobs.append((src, [CLANG + "++", "-x", "hip", "--offload-host-only",
                           "--offload-arch=gfx950", "-std=c++17", "-ffp-contract=off", *san,
                           f"-I{ROOT}/include", f"-I{CSRC}"]))
    objs = [os.path.join(BUILD, os.path.basename(src) + ".o") for src, _ in jobs]
    todo = [(cmd + ["-c", src, "-o", o]) for (src, cmd), o in zip(jobs, objs) if _stale(o, src)]
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        list(ex.map(_compile, todo))
    exe = os.path.join(BUILD, "host_check")
    if todo or not os.path.exists(exe):
        _compile([CLANG + "++", "-fsanitize=address,undefined", *objs, "-o", exe,
                  "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    return exe


def test_host_code_under_sanitizers():
    exe = _build()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=900, env=env)
    out = r.stdout + r.stderr
    assert "runtime error" not in out and "AddressSanitizer" not in out \
        and "LeakSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "0 failures" in out, out[-2000:]
