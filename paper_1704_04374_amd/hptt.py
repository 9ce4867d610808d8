"""Python binding of the C ABI in ``include/hptt.h``.

Argument marshalling only: every step of the transposition runs in the HIP
library ``libhptt.so`` built from ``csrc/``; PyTorch provides device memory
and streams.  There is no fallback: without the built library every call
raises ``HpttError``.

    plan = create_plan(perm=(1, 0), size_a=(8192, 8192), alpha=1.0, beta=0.0, dtype="f32")
    plan.exec(A, B)                       # A, B: flat CUDA tensors of numel elements
    B = transpose(A, (8192, 8192), (1, 0))
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libhptt.so")
MAX_DIMS = 16

DTYPES = {"f32": 0, "f64": 1}
KERNELS = {0: "auto", 1: "none", 2: "axpby", 3: "stream", 4: "tile", 5: "generic"}
KERNEL_IDS = {v: k for k, v in KERNELS.items()}
MODES = {0: "copy", 1: "scale", 2: "axpby"}

SUCCESS = 0
HIP_ERROR = 5
STATUS = {0: "HPTT_SUCCESS", 1: "HPTT_ERROR_INVALID_ARGUMENT", 2: "HPTT_ERROR_UNSUPPORTED",
          3: "HPTT_ERROR_OVERLAP", 4: "HPTT_ERROR_OUT_OF_MEMORY", 5: "HPTT_ERROR_HIP"}


class HpttError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {STATUS.get(status, status)}")
        self.status = status


class Options(ctypes.Structure):
    """hptt_options_t"""
    _fields_ = [("kernel", ctypes.c_int), ("run_a", ctypes.c_int32), ("run_b", ctypes.c_int32),
                ("max_vec", ctypes.c_int32), ("store_hint", ctypes.c_int32),
                ("load_hint", ctypes.c_int32), ("lds_pad", ctypes.c_int32),
                ("max_blocks", ctypes.c_int32), ("tile_order", ctypes.c_int32),
                ("exact_runs", ctypes.c_int32), ("row_passes", ctypes.c_int32),
                ("depth", ctypes.c_int32), ("min_tile", ctypes.c_int32),
                ("block", ctypes.c_int32), ("skew", ctypes.c_int32), ("shear", ctypes.c_int32),
                ("shared_runs", ctypes.c_int32), ("flat_runs", ctypes.c_int32),
                ("grid_order", ctypes.c_int32), ("direct_lds", ctypes.c_int32),
                ("xcd_group", ctypes.c_int32)]


class AutotuneReport(ctypes.Structure):
    """hptt_autotune_report_t"""
    _fields_ = [("candidates", ctypes.c_int32), ("timed", ctypes.c_int32),
                ("from_cache", ctypes.c_int32), ("flushed", ctypes.c_int32),
                ("own_mode", ctypes.c_int32), ("default_ms", ctypes.c_float),
                ("best_ms", ctypes.c_float), ("options", Options),
                ("finalists", ctypes.c_int32), ("confirmed", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {"candidates": self.candidates, "timed": self.timed,
                "from_cache": bool(self.from_cache), "flushed": bool(self.flushed),
                "own_mode": bool(self.own_mode), "default_ms": self.default_ms,
                "best_ms": self.best_ms, "finalists": self.finalists,
                "confirmed": self.confirmed,
                "options": {name: getattr(self.options, name) for name, _ in Options._fields_}}


class PlanInfo(ctypes.Structure):
    """hptt_plan_info_t"""
    _fields_ = [("ndim", ctypes.c_int32), ("size", ctypes.c_int64 * MAX_DIMS),
                ("perm", ctypes.c_int32 * MAX_DIMS), ("kernel", ctypes.c_int),
                ("numel", ctypes.c_int64), ("elem_bytes", ctypes.c_int32),
                ("run_a", ctypes.c_int64), ("run_b", ctypes.c_int64),
                ("dims_a", ctypes.c_int32), ("dims_b", ctypes.c_int32),
                ("vec_a", ctypes.c_int32), ("vec_b", ctypes.c_int32),
                ("lds_pitch", ctypes.c_int32), ("rows_per_pass", ctypes.c_int32),
                ("footprint_a", ctypes.c_int64), ("footprint_b", ctypes.c_int64),
                ("lds_bytes", ctypes.c_int32),
                ("tiles", ctypes.c_int64), ("grid", ctypes.c_int64), ("block", ctypes.c_int32),
                ("hints", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("tile_order", ctypes.c_int32), ("depth", ctypes.c_int32),
                ("shear", ctypes.c_int32), ("shared_runs", ctypes.c_int32),
                ("flat_runs", ctypes.c_int32), ("grid_order", ctypes.c_int32),
                ("direct_lds", ctypes.c_int32), ("xcd_group", ctypes.c_int32)]

    def as_dict(self) -> dict:
        n = self.ndim
        return {"ndim": n, "size": tuple(self.size[:n]), "perm": tuple(self.perm[:n]),
                "kernel": KERNELS[self.kernel], "numel": self.numel,
                "elem_bytes": self.elem_bytes, "run_a": self.run_a, "run_b": self.run_b,
                "dims_a": self.dims_a, "dims_b": self.dims_b, "vec_a": self.vec_a,
                "vec_b": self.vec_b, "lds_pitch": self.lds_pitch,
                "rows_per_pass": self.rows_per_pass, "footprint_a": self.footprint_a,
                "footprint_b": self.footprint_b, "lds_bytes": self.lds_bytes,
                "tiles": self.tiles, "grid": self.grid, "block": self.block,
                "hints": self.hints, "mode": MODES[self.mode],
                "tile_order": self.tile_order, "depth": self.depth, "shear": self.shear,
                "shared_runs": self.shared_runs, "flat_runs": self.flat_runs,
                "grid_order": self.grid_order, "direct_lds": self.direct_lds,
                "xcd_group": self.xcd_group}


# Every entry point declared in include/hptt.h and include/hptt_yardstick.h.
EXPORTS = ("hptt_create_plan", "hptt_create_plan_ex", "hptt_create_plan_outer",
           "hptt_create_plan_autotune", "hptt_autotune_candidates", "hptt_forget_wisdom",
           "hptt_exec", "hptt_destroy_plan",
           "hptt_plan_info", "hptt_describe_plan", "hptt_status_string",
           "hptt_last_hip_error", "hptt_load_kernels", "hptt_yardstick_copy",
           "hptt_yardstick_axpby",
           "hptt_yardstick_fill", "hptt_yardstick_read")


def _declare(lib: ctypes.CDLL, gpu: bool) -> ctypes.CDLL:
    i32p = ctypes.POINTER(ctypes.c_int32)
    i64p = ctypes.POINTER(ctypes.c_int64)
    vp = ctypes.c_void_p
    st = ctypes.c_int
    lib.hptt_create_plan.argtypes = [ctypes.POINTER(vp), i32p, ctypes.c_int32, i64p,
                                     ctypes.c_double, ctypes.c_double, ctypes.c_int]
    lib.hptt_create_plan_ex.argtypes = lib.hptt_create_plan.argtypes + [ctypes.POINTER(Options)]
    lib.hptt_create_plan_outer.argtypes = [ctypes.POINTER(vp), i32p, ctypes.c_int32, i64p, i64p,
                                           i64p, ctypes.c_double, ctypes.c_double, ctypes.c_int,
                                           ctypes.POINTER(Options)]
    lib.hptt_destroy_plan.argtypes = [vp]
    lib.hptt_plan_info.argtypes = [vp, ctypes.POINTER(PlanInfo)]
    lib.hptt_describe_plan.argtypes = [vp, ctypes.c_char_p, ctypes.c_size_t]
    lib.hptt_status_string.argtypes = [ctypes.c_int]
    lib.hptt_status_string.restype = ctypes.c_char_p
    for f in ("hptt_create_plan", "hptt_create_plan_ex", "hptt_create_plan_outer",
              "hptt_destroy_plan", "hptt_plan_info", "hptt_describe_plan"):
        getattr(lib, f).restype = st
    if gpu:
        lib.hptt_autotune_candidates.argtypes = [i32p, ctypes.c_int32, i64p, i64p, i64p,
                                                 ctypes.c_double, ctypes.c_double, ctypes.c_int,
                                                 ctypes.POINTER(Options), ctypes.c_int32]
        lib.hptt_autotune_candidates.restype = ctypes.c_int32
        lib.hptt_create_plan_autotune.argtypes = [ctypes.POINTER(vp), i32p, ctypes.c_int32, i64p,
                                                  i64p, i64p, ctypes.c_double, ctypes.c_double,
                                                  ctypes.c_int, vp, vp, vp, ctypes.c_double,
                                                  ctypes.POINTER(AutotuneReport)]
        lib.hptt_create_plan_autotune.restype = st
        lib.hptt_forget_wisdom.restype = st
        lib.hptt_exec.argtypes = [vp, vp, vp, vp]
        lib.hptt_exec.restype = st
        lib.hptt_last_hip_error.restype = ctypes.c_int32
        lib.hptt_load_kernels.restype = st
        lib.hptt_yardstick_copy.argtypes = [vp, vp, ctypes.c_size_t, vp]
        lib.hptt_yardstick_axpby.argtypes = [ctypes.c_int, ctypes.c_double, vp, ctypes.c_double,
                                             vp, ctypes.c_size_t, vp]
        lib.hptt_yardstick_fill.argtypes = [vp, ctypes.c_size_t, ctypes.c_uint32, vp]
        lib.hptt_yardstick_read.argtypes = [vp, ctypes.c_size_t, vp, vp]
        for f in ("hptt_yardstick_copy", "hptt_yardstick_axpby", "hptt_yardstick_fill",
                  "hptt_yardstick_read"):
            getattr(lib, f).restype = st
    return lib


_lib = None


def library() -> ctypes.CDLL:
    """The loaded ``libhptt.so``; raises HpttError if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise HpttError(-1, f"{LIB_PATH} is missing; run paper_1704_04374_amd.build")
        _lib = _declare(ctypes.CDLL(LIB_PATH), gpu=True)
    return _lib


def load_kernels() -> None:
    """hptt_load_kernels: load the library's GPU code onto the current device."""
    st = library().hptt_load_kernels()
    if st == HIP_ERROR:
        raise HpttError(st, f"hptt_load_kernels (hipError {library().hptt_last_hip_error()})")
    _check(st, "hptt_load_kernels")


def load_plan_api(path: str) -> ctypes.CDLL:
    """Load another library that exports the plan half of the ABI (for tests)."""
    return _declare(ctypes.CDLL(path), gpu=False)


def _dtype_id(dtype) -> int:
    if isinstance(dtype, str):
        return DTYPES[dtype]
    import torch
    if dtype == torch.float32:
        return 0
    if dtype == torch.float64:
        return 1
    raise TypeError(f"unsupported dtype {dtype}")


def _check(status: int, what: str):
    if status != SUCCESS:
        raise HpttError(status, what)


class Plan:
    """A plan for Eq. (1): perm[k] is the A index at position k of B (0-based),
    tensors are Fortran-ordered (first index fastest).  With ``outer_size_a``
    (A's index order) and/or ``outer_size_b`` (B's index order) A and B are
    sub-tensors of larger tensors of those extents (Fig. 3)."""

    def __init__(self, perm, size_a, alpha: float = 1.0, beta: float = 0.0, dtype="f32",
                 options: Options | None = None, lib: ctypes.CDLL | None = None,
                 outer_size_a=None, outer_size_b=None, **knobs):
        self._lib = lib if lib is not None else library()
        self._handle = None
        n = len(perm)
        if len(size_a) != n:
            raise ValueError("perm and size_a differ in length")
        self.perm = tuple(int(p) for p in perm)
        self.size_a = tuple(int(s) for s in size_a)
        self.alpha, self.beta = float(alpha), float(beta)
        self.dtype = dtype if isinstance(dtype, str) else {0: "f32", 1: "f64"}[_dtype_id(dtype)]
        pm = (ctypes.c_int32 * max(n, 1))(*self.perm)
        sz = (ctypes.c_int64 * max(n, 1))(*self.size_a)
        handle = ctypes.c_void_p()
        if knobs:
            options = options or Options()
            for k, v in knobs.items():
                setattr(options, k, KERNEL_IDS[v] if k == "kernel" and isinstance(v, str) else v)
        self.outer_size_a = None if outer_size_a is None else tuple(int(x) for x in outer_size_a)
        self.outer_size_b = None if outer_size_b is None else tuple(int(x) for x in outer_size_b)
        if self.outer_size_a is not None or self.outer_size_b is not None:
            oa = None if self.outer_size_a is None else (ctypes.c_int64 * n)(*self.outer_size_a)
            ob = None if self.outer_size_b is None else (ctypes.c_int64 * n)(*self.outer_size_b)
            for o in (self.outer_size_a, self.outer_size_b):
                if o is not None and len(o) != n:
                    raise ValueError("outer sizes need one extent per index")
            st = self._lib.hptt_create_plan_outer(ctypes.byref(handle), pm, n, sz, oa, ob,
                                                  self.alpha, self.beta, DTYPES[self.dtype],
                                                  None if options is None else ctypes.byref(options))
        elif options is None:
            st = self._lib.hptt_create_plan(ctypes.byref(handle), pm, n, sz, self.alpha,
                                            self.beta, DTYPES[self.dtype])
        else:
            st = self._lib.hptt_create_plan_ex(ctypes.byref(handle), pm, n, sz, self.alpha,
                                               self.beta, DTYPES[self.dtype], ctypes.byref(options))
        _check(st, "hptt_create_plan")
        self._handle = handle

    @property
    def handle(self) -> ctypes.c_void_p:
        return self._handle

    @property
    def info(self) -> dict:
        out = PlanInfo()
        _check(self._lib.hptt_plan_info(self._handle, ctypes.byref(out)), "hptt_plan_info")
        return out.as_dict()

    def describe(self) -> str:
        buf = ctypes.create_string_buffer(512)
        _check(self._lib.hptt_describe_plan(self._handle, buf, len(buf)), "hptt_describe_plan")
        return buf.value.decode()

    @property
    def numel(self) -> int:
        n = 1
        for s in self.size_a:
            n *= s
        return n

    @property
    def size_b(self) -> tuple:
        return tuple(self.size_a[p] for p in self.perm)

    def exec(self, A, B, stream=None):
        """Queue B <- alpha*A + beta*B (permuted) on `stream` (default: torch's
        current stream).  A and B are CUDA tensors (or raw device pointers)."""
        a = A if isinstance(A, int) else A.data_ptr()
        b = B if isinstance(B, int) else B.data_ptr()
        if not isinstance(A, int):
            self._check_tensor(A, "A")
            self._check_tensor(B, "B")
        if stream is None:
            import torch
            stream = torch.cuda.current_stream().cuda_stream
        elif not isinstance(stream, int):
            stream = stream.cuda_stream
        st = self._lib.hptt_exec(self._handle, ctypes.c_void_p(a), ctypes.c_void_p(b),
                                 ctypes.c_void_p(stream))
        if st == HIP_ERROR:
            raise HpttError(st, f"hptt_exec (hipError {self._lib.hptt_last_hip_error()})")
        _check(st, "hptt_exec")

    def launcher(self, A_ptr: int, B_ptr: int, stream: int):
        """A zero-argument callable that queues this plan on fixed device
        pointers and stream with no per-call checks (for timing loops)."""
        f = self._lib.hptt_exec
        h, a, b, s = self._handle, ctypes.c_void_p(A_ptr), ctypes.c_void_p(B_ptr), ctypes.c_void_p(stream)

        def run():
            st = f(h, a, b, s)
            if st != SUCCESS:
                raise HpttError(st, "hptt_exec")
        return run

    def _check_tensor(self, t, name):
        if not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
        info = self.info
        need = info["footprint_a"] if name == "A" else info["footprint_b"]
        if not t.is_contiguous() or t.numel() < need or (
                self.outer_size_a is None and self.outer_size_b is None and t.numel() != need):
            raise ValueError(f"{name} must be contiguous and cover {need} elements")
        if _dtype_id(t.dtype) != DTYPES[self.dtype]:
            raise ValueError(f"{name} has dtype {t.dtype}, plan is {self.dtype}")

    def __del__(self):
        if getattr(self, "_handle", None) is not None and self._handle.value:
            self._lib.hptt_destroy_plan(self._handle)
            self._handle = None


def create_plan(perm, size_a, alpha=1.0, beta=0.0, dtype="f32", **knobs) -> Plan:
    return Plan(perm, size_a, alpha, beta, dtype, **knobs)


def transpose(A, size_a, perm, alpha=1.0, beta=0.0, B=None, **knobs):
    """Return B with B_{perm} = alpha*A + beta*B for a flat CUDA tensor A
    holding a Fortran-ordered tensor of extents size_a."""
    import torch
    plan = Plan(perm, size_a, alpha, beta, A.dtype, **knobs)
    if B is None:
        if beta != 0:
            raise ValueError("beta != 0 needs B")
        B = torch.empty_like(A)
    plan.exec(A, B)
    return B


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def yardstick_copy(src, dst, nbytes: int, stream=None):
    _check(library().hptt_yardstick_copy(ctypes.c_void_p(src.data_ptr()),
                                         ctypes.c_void_p(dst.data_ptr()), nbytes,
                                         ctypes.c_void_p(_stream(stream))), "hptt_yardstick_copy")


def yardstick_axpby(dtype, alpha, x, beta, y, n: int, stream=None):
    _check(library().hptt_yardstick_axpby(_dtype_id(dtype), float(alpha),
                                          ctypes.c_void_p(x.data_ptr()), float(beta),
                                          ctypes.c_void_p(y.data_ptr()), n,
                                          ctypes.c_void_p(_stream(stream))), "hptt_yardstick_axpby")


def yardstick_fill(buf, nbytes: int, value: int = 0, stream=None):
    _check(library().hptt_yardstick_fill(ctypes.c_void_p(buf.data_ptr()), nbytes, value,
                                         ctypes.c_void_p(_stream(stream))), "hptt_yardstick_fill")


def yardstick_read(buf, nbytes: int, sink, stream=None):
    _check(library().hptt_yardstick_read(ctypes.c_void_p(buf.data_ptr()), nbytes,
                                         ctypes.c_void_p(sink.data_ptr()),
                                         ctypes.c_void_p(_stream(stream))), "hptt_yardstick_read")


def _sizes(values, n):
    return None if values is None else (ctypes.c_int64 * n)(*[int(x) for x in values])


def autotune_candidates(perm, size_a, alpha=1.0, beta=0.0, dtype="f32", outer_size_a=None,
                        outer_size_b=None, max_options: int = 256) -> list:
    """The knobs hptt_create_plan_autotune would time, in its order."""
    n = len(perm)
    out = (Options * max_options)()
    cnt = library().hptt_autotune_candidates(
        (ctypes.c_int32 * n)(*perm), n, (ctypes.c_int64 * n)(*size_a), _sizes(outer_size_a, n),
        _sizes(outer_size_b, n), float(alpha), float(beta), _dtype_id(dtype), out, max_options)
    if cnt < 0:
        raise HpttError(-cnt, "hptt_autotune_candidates")
    return [{name: getattr(out[i], name) for name, _ in Options._fields_}
            for i in range(min(cnt, max_options))]


def autotune_plan(perm, size_a, A, B, alpha=1.0, beta=0.0, dtype="f32", timeout=1.0,
                  outer_size_a=None, outer_size_b=None, stream=None):
    """A plan tuned on the device tensors A and B (which keep their values)
    within ``timeout`` seconds; returns (Plan, report dict)."""
    plan = Plan(perm, size_a, alpha, beta, dtype, outer_size_a=outer_size_a,
                outer_size_b=outer_size_b)
    plan._check_tensor(A, "A")   # the tuner launches on A and B: check them first
    plan._check_tensor(B, "B")
    n = len(plan.perm)
    handle = ctypes.c_void_p()
    rep = AutotuneReport()
    st = plan._lib.hptt_create_plan_autotune(
        ctypes.byref(handle), (ctypes.c_int32 * n)(*plan.perm), n,
        (ctypes.c_int64 * n)(*plan.size_a), _sizes(plan.outer_size_a, n),
        _sizes(plan.outer_size_b, n), plan.alpha, plan.beta, DTYPES[plan.dtype],
        ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(B.data_ptr()),
        ctypes.c_void_p(_stream(stream)), float(timeout), ctypes.byref(rep))
    _check(st, "hptt_create_plan_autotune")
    plan._lib.hptt_destroy_plan(plan._handle)
    plan._handle = handle
    return plan, rep.as_dict()


def forget_wisdom():
    _check(library().hptt_forget_wisdom(), "hptt_forget_wisdom")
