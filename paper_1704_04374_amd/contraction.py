"""ctypes binding of the contraction library (include/hptt_contract.h):
C = alpha * A . B + beta * C on Fortran-ordered device tensors, by
transposition - GEMM - transposition.  Argument marshalling only; the
workspace is device memory from torch's allocator."""
from __future__ import annotations

import ctypes
import os

from . import hptt

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhptt_contract.so")

EXPORTS = ("hptt_contraction_create", "hptt_contraction_destroy", "hptt_contraction_info",
           "hptt_contraction_describe", "hptt_contraction_exec",
           "hptt_contraction_exec_no_alloc", "hptt_contraction_last_blas_status")

# the device array hptt_contraction_exec_no_alloc works in, and rocBLAS's share of it
STATIC_BYTES = 64 << 20
STATIC_BLAS_BYTES = 16 << 20


class ContractionInfo(ctypes.Structure):
    """hptt_contraction_info_t"""
    _fields_ = [("transpose_a", ctypes.c_int32), ("transpose_b", ctypes.c_int32),
                ("transpose_c", ctypes.c_int32), ("swap", ctypes.c_int32),
                ("op_p", ctypes.c_int32), ("op_q", ctypes.c_int32),
                ("gemm_m", ctypes.c_int64), ("gemm_n", ctypes.c_int64),
                ("gemm_k", ctypes.c_int64), ("batch", ctypes.c_int64),
                ("ld_p", ctypes.c_int64), ("ld_q", ctypes.c_int64), ("ld_c", ctypes.c_int64),
                ("stride_p", ctypes.c_int64), ("stride_q", ctypes.c_int64),
                ("stride_c", ctypes.c_int64), ("modes_x", ctypes.c_char * 17),
                ("modes_y", ctypes.c_char * 17), ("modes_k", ctypes.c_char * 17),
                ("modes_l", ctypes.c_char * 17), ("workspace_bytes", ctypes.c_int64),
                ("flops", ctypes.c_double), ("bytes_transposed", ctypes.c_double)]

    def as_dict(self) -> dict:
        return {name: (v.decode() if isinstance(v, bytes) else v)
                for name, v in ((n, getattr(self, n)) for n, _ in self._fields_)}


_lib = None


def library() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise hptt.HpttError(-1, f"{LIB_PATH} is missing; run paper_1704_04374_amd.build")
        hptt.library()  # libhptt.so first, for its symbols
        lib = ctypes.CDLL(LIB_PATH)
        vp, i64p, st = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64), ctypes.c_int
        lib.hptt_contraction_create.argtypes = [ctypes.POINTER(vp), ctypes.c_int, ctypes.c_double,
                                                ctypes.c_double, ctypes.c_char_p, i64p,
                                                ctypes.c_char_p, i64p, ctypes.c_char_p]
        lib.hptt_contraction_destroy.argtypes = [vp]
        lib.hptt_contraction_info.argtypes = [vp, ctypes.POINTER(ContractionInfo)]
        lib.hptt_contraction_describe.argtypes = [vp, ctypes.c_char_p, ctypes.c_size_t]
        lib.hptt_contraction_exec.argtypes = [vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        lib.hptt_contraction_exec_no_alloc.argtypes = [vp, vp, vp, vp, vp]
        lib.hptt_contraction_last_blas_status.restype = ctypes.c_int32
        for f in ("hptt_contraction_create", "hptt_contraction_destroy", "hptt_contraction_info",
                  "hptt_contraction_describe", "hptt_contraction_exec",
                  "hptt_contraction_exec_no_alloc"):
            getattr(lib, f).restype = st
        _lib = lib
    return _lib


class Contraction:
    """C[modes_c] = alpha * sum A[modes_a] B[modes_b] + beta * C[modes_c]
    (one character per mode, first mode fastest)."""

    def __init__(self, modes_c: str, modes_a: str, size_a, modes_b: str, size_b,
                 alpha: float = 1.0, beta: float = 0.0, dtype="f64"):
        self._lib = library()
        self._handle = None
        self.modes_a, self.modes_b, self.modes_c = modes_a, modes_b, modes_c
        self.size_a = tuple(int(s) for s in size_a)
        self.size_b = tuple(int(s) for s in size_b)
        if len(self.size_a) != len(modes_a) or len(self.size_b) != len(modes_b):
            raise ValueError("one extent per mode")
        self.alpha, self.beta = float(alpha), float(beta)
        self.dtype = dtype if isinstance(dtype, str) else {0: "f32", 1: "f64"}[hptt._dtype_id(dtype)]
        ext = dict(zip(modes_a, self.size_a))
        ext.update(zip(modes_b, self.size_b))
        self.size_c = tuple(ext.get(m, 0) for m in modes_c)
        handle = ctypes.c_void_p()
        sa = (ctypes.c_int64 * max(1, len(self.size_a)))(*self.size_a)
        sb = (ctypes.c_int64 * max(1, len(self.size_b)))(*self.size_b)
        st = self._lib.hptt_contraction_create(ctypes.byref(handle), hptt.DTYPES[self.dtype],
                                               self.alpha, self.beta, modes_a.encode(), sa,
                                               modes_b.encode(), sb, modes_c.encode())
        hptt._check(st, "hptt_contraction_create")
        self._handle = handle
        self._workspace = None

    @property
    def info(self) -> dict:
        out = ContractionInfo()
        hptt._check(self._lib.hptt_contraction_info(self._handle, ctypes.byref(out)),
                    "hptt_contraction_info")
        return out.as_dict()

    def describe(self) -> str:
        buf = ctypes.create_string_buffer(512)
        hptt._check(self._lib.hptt_contraction_describe(self._handle, buf, len(buf)),
                    "hptt_contraction_describe")
        return buf.value.decode()

    def workspace(self):
        """The device workspace this plan executes with (allocated once)."""
        import torch
        need = self.info["workspace_bytes"]
        if need and (self._workspace is None or self._workspace.numel() < need):
            self._workspace = torch.empty(need, dtype=torch.uint8, device="cuda")
        return self._workspace

    def _check_tensors(self, A, B, C):
        for t, name, n in ((A, "A", self.size_a), (B, "B", self.size_b), (C, "C", self.size_c)):
            numel = 1
            for s in n:
                numel *= s
            if not t.is_cuda or not t.is_contiguous() or t.numel() != numel:
                raise ValueError(f"{name} must be a contiguous device tensor of {numel} elements")
            if hptt._dtype_id(t.dtype) != hptt.DTYPES[self.dtype]:
                raise ValueError(f"{name} has dtype {t.dtype}, plan is {self.dtype}")

    def _raise(self, st, what):
        if st == hptt.HIP_ERROR:
            raise hptt.HpttError(st, f"{what} (hipError {hptt.library().hptt_last_hip_error()}, "
                                     f"rocBLAS status "
                                     f"{self._lib.hptt_contraction_last_blas_status()})")
        hptt._check(st, what)

    def exec(self, A, B, C, stream=None):
        """Queue the contraction on `stream` (default: torch's current one)."""
        self._check_tensors(A, B, C)
        ws = self.workspace()
        st = self._lib.hptt_contraction_exec(
            self._handle, ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(B.data_ptr()),
            ctypes.c_void_p(C.data_ptr()), ctypes.c_void_p(0 if ws is None else ws.data_ptr()),
            0 if ws is None else ws.numel(), ctypes.c_void_p(hptt._stream(stream)))
        self._raise(st, "hptt_contraction_exec")

    def exec_no_alloc(self, A, B, C, stream=None):
        """Queue the contraction on `stream` with the library's own device
        array as the workspace (hptt_contraction_exec_no_alloc): nothing is
        allocated; calls that overlap on one device race."""
        self._check_tensors(A, B, C)
        st = self._lib.hptt_contraction_exec_no_alloc(
            self._handle, ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(B.data_ptr()),
            ctypes.c_void_p(C.data_ptr()), ctypes.c_void_p(hptt._stream(stream)))
        self._raise(st, "hptt_contraction_exec_no_alloc")

    def __del__(self):
        if getattr(self, "_handle", None) is not None and self._handle.value:
            self._lib.hptt_contraction_destroy(self._handle)
            self._handle = None
