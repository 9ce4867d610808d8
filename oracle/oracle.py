"""Python binding of the C oracle for Eq. (1) of the HPTT paper (Section 1).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test-suite, the smoke check
of the entry module and the CPU-baseline leg of the benchmark may import this
module.  It never touches the GPU library and works on host numpy arrays.

Conventions (see the header of ``oracle.c``): tensors are flat arrays in the
Fortran layout of Section 1; ``perm[k]`` is the A index at position k of B
(0-based, Fig. 3b and Table 1); alpha and beta are rounded once to the tensor
dtype before use.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# -ffp-contract=off: no fused multiply-add, so every product and the sum are
# rounded separately, as in the reading stated in oracle.c.
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-std=c99"]


def compile_source(src: str, out: str) -> str:
    """Compile an oracle source file into a shared library at ``out``."""
    tmp = f"{out}.tmp{os.getpid()}"  # one per process: test workers may build at once
    subprocess.check_call(["gcc", *CFLAGS, src, "-o", tmp])
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` beside it."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        compile_source(_SRC, _LIB)
    return _LIB


class OracleLib:
    """The oracle entry points of one compiled library."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        i64p = ctypes.POINTER(ctypes.c_int64)
        i32p = ctypes.POINTER(ctypes.c_int32)
        vp = ctypes.c_void_p
        lib.oracle_size_b.argtypes = [ctypes.c_int, i64p, i32p, i64p]
        lib.oracle_transpose_f32.argtypes = [ctypes.c_int, i64p, i32p, ctypes.c_float,
                                             ctypes.c_float, vp, vp]
        lib.oracle_transpose_f64.argtypes = [ctypes.c_int, i64p, i32p, ctypes.c_double,
                                             ctypes.c_double, vp, vp]
        lib.oracle_transpose_outer_f32.argtypes = [ctypes.c_int, i64p, i32p, i64p, i64p,
                                                   ctypes.c_float, ctypes.c_float, vp, vp]
        lib.oracle_transpose_outer_f64.argtypes = [ctypes.c_int, i64p, i32p, i64p, i64p,
                                                   ctypes.c_double, ctypes.c_double, vp, vp]
        lib.oracle_sample_f32.argtypes = [ctypes.c_int, i64p, i32p, ctypes.c_float,
                                          ctypes.c_float, vp, vp, ctypes.c_int64, i64p, vp]
        lib.oracle_sample_f64.argtypes = [ctypes.c_int, i64p, i32p, ctypes.c_double,
                                          ctypes.c_double, vp, vp, ctypes.c_int64, i64p, vp]
        for f in ("oracle_size_b", "oracle_transpose_f32", "oracle_transpose_f64",
                  "oracle_transpose_outer_f32", "oracle_transpose_outer_f64",
                  "oracle_sample_f32", "oracle_sample_f64"):
            getattr(lib, f).restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def size_b(self, size_a, perm):
        """Compact extents of B: ``sizeB[k] = sizeA[perm[k]]`` (Fig. 3b)."""
        n, sz, pm = _problem(size_a, perm)
        out = (ctypes.c_int64 * n)()
        err = self.lib.oracle_size_b(n, sz, pm, out)
        if err:
            raise ValueError(f"invalid problem (oracle error {err})")
        return tuple(out)

    def transpose(self, A: np.ndarray, size_a, perm, alpha: float = 1.0, beta: float = 0.0,
                  B: np.ndarray | None = None) -> np.ndarray:
        """Return B after Eq. (1).  ``A`` and ``B`` are flat Fortran-layout
        arrays of dtype float32 or float64.  ``B`` (the prior contents, needed
        only when beta != 0) is not modified; a new array is returned."""
        dtype = A.dtype
        if dtype not in (np.float32, np.float64):
            raise TypeError("oracle supports float32 and float64")
        numel = _numel(size_a)
        _check_arrays(A, B, numel, dtype)
        n, sz, pm = _problem(size_a, perm)
        if B is None:
            if beta != 0:
                raise ValueError("beta != 0 needs the prior B")
            out = np.zeros(numel, dtype=dtype)
        else:
            out = B.copy()
        if dtype == np.float32:
            err = self.lib.oracle_transpose_f32(n, sz, pm, float(np.float32(alpha)),
                                                float(np.float32(beta)),
                                                A.ctypes.data, out.ctypes.data)
        else:
            err = self.lib.oracle_transpose_f64(n, sz, pm, float(alpha), float(beta),
                                                A.ctypes.data, out.ctypes.data)
        if err:
            raise ValueError(f"invalid problem (oracle error {err})")
        return out

    def transpose_outer(self, A: np.ndarray, size_a, perm, outer_a, outer_b,
                        alpha: float = 1.0, beta: float = 0.0,
                        B: np.ndarray | None = None) -> np.ndarray:
        """Eq. (1) on sub-tensors (Fig. 3).  ``A`` and ``B`` are flat arrays
        whose first elements are the sub-tensors' first elements, with the
        Fortran strides of the enclosing extents ``outer_a`` (A's index
        order) and ``outer_b`` (B's index order); each must cover its
        sub-tensor's footprint.  ``B`` (zeros if None) is not modified; a new
        array is returned in which only the sub-tensor's elements changed."""
        dtype = A.dtype
        if dtype not in (np.float32, np.float64):
            raise TypeError("oracle supports float32 and float64")
        n, sz, pm = _problem(size_a, perm)
        if len(outer_a) != n or len(outer_b) != n:
            raise ValueError("outer sizes must have N entries")
        size_b = [size_a[p] for p in perm]
        if A.ndim != 1 or A.size < footprint(size_a, outer_a) or not A.flags.c_contiguous:
            raise ValueError("A must be a flat contiguous array covering the sub-tensor")
        if B is None:
            out = np.zeros(footprint(size_b, outer_b), dtype=dtype)
        else:
            out = B.copy()
        if out.ndim != 1 or out.size < footprint(size_b, outer_b) or out.dtype != dtype:
            raise ValueError("B must be a flat array covering the sub-tensor")
        oa = (ctypes.c_int64 * n)(*[int(x) for x in outer_a])
        ob = (ctypes.c_int64 * n)(*[int(x) for x in outer_b])
        if dtype == np.float32:
            err = self.lib.oracle_transpose_outer_f32(n, sz, pm, oa, ob, float(np.float32(alpha)),
                                                      float(np.float32(beta)), A.ctypes.data,
                                                      out.ctypes.data)
        else:
            err = self.lib.oracle_transpose_outer_f64(n, sz, pm, oa, ob, float(alpha),
                                                      float(beta), A.ctypes.data, out.ctypes.data)
        if err:
            raise ValueError(f"invalid problem (oracle error {err})")
        return out

    def sample(self, A: np.ndarray, size_a, perm, alpha: float, beta: float,
               B_in: np.ndarray | None, offsets_b: np.ndarray) -> np.ndarray:
        """Expected B values at the given B offsets, computed one element at
        a time (for tensors too large to transpose whole on the CPU)."""
        dtype = A.dtype
        numel = _numel(size_a)
        _check_arrays(A, B_in, numel, dtype)
        if beta != 0 and B_in is None:
            raise ValueError("beta != 0 needs the prior B")
        offs = np.ascontiguousarray(offsets_b, dtype=np.int64)
        out = np.empty(offs.size, dtype=dtype)
        n, sz, pm = _problem(size_a, perm)
        bptr = None if B_in is None else B_in.ctypes.data
        op = offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
        if dtype == np.float32:
            err = self.lib.oracle_sample_f32(n, sz, pm, float(np.float32(alpha)),
                                             float(np.float32(beta)), A.ctypes.data, bptr,
                                             offs.size, op, out.ctypes.data)
        else:
            err = self.lib.oracle_sample_f64(n, sz, pm, float(alpha), float(beta),
                                             A.ctypes.data, bptr, offs.size, op,
                                             out.ctypes.data)
        if err:
            raise ValueError(f"invalid problem or offset (oracle error {err})")
        return out


def footprint(size, outer) -> int:
    """Elements from a sub-tensor's first to its last element, inclusive,
    in an enclosing Fortran-ordered tensor of extents ``outer``."""
    if any(int(x) == 0 for x in size):
        return 0
    span, stride = 1, 1
    for n, o in zip(size, outer):
        span += (int(n) - 1) * stride
        stride *= int(o)
    return span


def _numel(size_a) -> int:
    n = 1
    for s in size_a:
        n *= int(s)
    return n


def _problem(size_a, perm):
    n = len(size_a)
    if len(perm) != n:
        raise ValueError("perm and size_a differ in length")
    sz = (ctypes.c_int64 * n)(*[int(s) for s in size_a])
    pm = (ctypes.c_int32 * n)(*[int(p) for p in perm])
    return n, sz, pm


def _check_arrays(A, B, numel, dtype):
    if A.dtype != dtype or A.ndim != 1 or A.size != numel or not A.flags.c_contiguous:
        raise ValueError("A must be a flat contiguous array of numel elements")
    if B is not None and (B.dtype != dtype or B.ndim != 1 or B.size != numel
                          or not B.flags.c_contiguous):
        raise ValueError("B must be a flat contiguous array of numel elements")


_default = None


def default() -> OracleLib:
    """The oracle built from ``oracle.c`` (compiled on first use)."""
    global _default
    if _default is None:
        _default = OracleLib(build(force=False))
    return _default


def size_b(size_a, perm):
    return default().size_b(size_a, perm)


def transpose(A, size_a, perm, alpha=1.0, beta=0.0, B=None):
    return default().transpose(A, size_a, perm, alpha, beta, B)


def sample(A, size_a, perm, alpha, beta, B_in, offsets_b):
    return default().sample(A, size_a, perm, alpha, beta, B_in, offsets_b)


def transpose_outer(A, size_a, perm, outer_a, outer_b, alpha=1.0, beta=0.0, B=None):
    return default().transpose_outer(A, size_a, perm, outer_a, outer_b, alpha, beta, B)
