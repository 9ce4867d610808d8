"""ctypes wrapper of the test-only host emulator (see emulate.cpp)."""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def library():
    global _lib
    if _lib is None:
        srcs = [os.path.join(_build.HERE, "emulate.cpp")] + [
            os.path.join(_build.CSRC, f) for f in os.listdir(_build.CSRC)]
        if not os.path.exists(_build.LIB) or any(
                os.path.getmtime(s) > os.path.getmtime(_build.LIB) for s in srcs):
            _build.build()
        from paper_1704_04374_amd.hptt import load_plan_api
        lib = load_plan_api(_build.LIB)
        lib.hptt_emulate_exec.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_char_p, ctypes.c_size_t,
                                          ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
        lib.hptt_emulate_exec.restype = ctypes.c_int64
        lib.hptt_emulate_check_fastdiv.argtypes = [ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64]
        lib.hptt_emulate_check_fastdiv.restype = ctypes.c_int64
        _lib = lib
    return _lib


def plan(perm, size_a, alpha=1.0, beta=0.0, dtype="f32", **knobs):
    from paper_1704_04374_amd.hptt import Plan
    return Plan(perm, size_a, alpha, beta, dtype, lib=library(), **knobs)


VARIANTS = {"fast": 0, "shifted": 1, "general": 2}


def run(p, A=None, B=None, va=0, vb=0, counts=False, block_stride=1, mis_a=0, mis_b=0,
        variant=None):
    """Emulate hptt_exec; B is updated in place.  mis_a/mis_b: element offsets
    of the base pointers from the 16-byte grid (tile kernel); variant:
    "general" (any plan) or "shifted" (plans the fast variant serves) runs the
    tile kernel in that variant instead of the one hptt_exec would launch.
    Returns (errors, msg, counts)."""
    lib = library()
    cnt = np.zeros(p.info["footprint_b"], dtype=np.uint8) if counts else None
    msg = ctypes.create_string_buffer(512)
    err = lib.hptt_emulate_exec(p.handle, None if A is None else A.ctypes.data,
                                None if B is None else B.ctypes.data, va, vb,
                                None if cnt is None else cnt.ctypes.data, block_stride, msg,
                                len(msg), mis_a, mis_b,
                                -1 if variant is None else VARIANTS[variant])
    return err, msg.value.decode(), cnt
