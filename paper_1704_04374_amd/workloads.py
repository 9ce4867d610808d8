"""Seeded synthetic workloads for the transposition of Eq. (1).

This module only describes problems and draws their input values; it holds
none of the transposition's arithmetic, so both the GPU path and the CPU
oracle may use it.  The five named workloads stand in for the paper's
benchmark of 57 transpositions of 2-D to 6-D tensors of about 200 MB each
(Section 4), whose case list the paper does not print: they span 2-D to 6-D,
fp32 and fp64, beta = 0 and beta != 0, and stride-1 moved and kept.

Values are uniform in [-1, 1): ``torch.rand`` in the tensor dtype, times 2,
minus 1, which is exact in that dtype (fp32 draws are multiples of 2^-24,
fp64 draws multiples of 2^-53), so no value is subnormal.
"""
from __future__ import annotations

from dataclasses import dataclass
from math import prod

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str              # "f32" or "f64"
    size_a: tuple           # extents of A, Fortran order (first index fastest)
    perm: tuple             # perm[k] = A index at position k of B (0-based)
    alpha: float
    beta: float
    seed_a: int
    seed_b: int | None      # prior B contents (only when beta != 0)
    # Sub-tensors (Fig. 3): extents of the enclosing tensors (A's / B's index
    # order) and the sub-tensors' first multi-indices in them; None = compact.
    outer_a: tuple | None = None
    outer_b: tuple | None = None
    start_a: tuple | None = None
    start_b: tuple | None = None
    # plan options ((name, value), ...) the benchmark builds the plan with;
    # () = the quick path's own choices (every benchmark workload)
    knobs: tuple = ()

    @property
    def numel(self) -> int:
        return prod(self.size_a)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 8

    @property
    def size_b(self) -> tuple:
        return tuple(self.size_a[p] for p in self.perm)

    @property
    def tensor_bytes(self) -> int:
        """S of Eq. (2): bytes of one tensor."""
        return self.numel * self.elem_bytes

    @property
    def lam(self) -> int:
        """lambda of Eq. (2): 2 when B is only written, 3 when it is updated."""
        return 2 if self.beta == 0 else 3

    @property
    def moved_bytes(self) -> int:
        """lambda * S: bytes an ideal implementation moves through memory."""
        return self.lam * self.tensor_bytes

    @property
    def parent_numel_a(self) -> int:
        return prod(self.outer_a) if self.outer_a else self.numel

    @property
    def parent_numel_b(self) -> int:
        return prod(self.outer_b) if self.outer_b else self.numel

    @property
    def offset_a(self) -> int:
        """Element offset of A's sub-tensor in its enclosing tensor."""
        return _fortran_offset(self.start_a, self.outer_a) if self.start_a else 0

    @property
    def offset_b(self) -> int:
        return _fortran_offset(self.start_b, self.outer_b) if self.start_b else 0

    def describe(self) -> str:
        d = (f"{self.name}: {self.dtype} A{self.size_a} perm{list(self.perm)} -> "
             f"B{self.size_b}, alpha={self.alpha}, beta={self.beta}")
        if self.outer_a:
            d += f", A inside {self.outer_a} at {self.start_a}"
        if self.outer_b:
            d += f", B inside {self.outer_b} at {self.start_b}"
        return d


WORKLOADS = [
    Workload("transpose3d_48x40x32_f32", "f32", (48, 40, 32), (2, 0, 1), 1.0, 0.0, 0, None),
    Workload("transpose2d_8192x8192_f32", "f32", (8192, 8192), (1, 0), 1.0, 0.0, 1, None),
    Workload("transpose6d_24x20x16x24x18x20_f32", "f32", (24, 20, 16, 24, 18, 20),
             (5, 2, 0, 4, 1, 3), 1.5, 0.0, 2, None),
    Workload("transpose4d_96x96x96x96_keep1_f64", "f64", (96, 96, 96, 96), (0, 3, 2, 1),
             2.0, 0.5, 3, 4),
    Workload("transpose5d_3x2x640x480x96_f32", "f32", (3, 2, 640, 480, 96), (4, 2, 0, 3, 1),
             1.0, 1.0, 5, 6),
]

# Sub-tensor workloads (Section 3.1, Fig. 3): transpose-and-compact and its
# reverse, transpose-and-scatter, on a half of an 8192 x 8192 fp32 matrix.
SUBTENSOR_WORKLOADS = [
    Workload("compact_4096x8192_of_8192x8192_f32", "f32", (4096, 8192), (1, 0), 1.0, 0.0, 7,
             None, outer_a=(8192, 8192), start_a=(2048, 0)),
    Workload("scatter_4096x8192_into_8192x8192_f32", "f32", (4096, 8192), (1, 0), 1.0, 0.0, 8,
             None, outer_b=(8192, 8192), start_b=(0, 2048)),
]

# Diagnostic workload for profiling, not a benchmark line: the 6-D fp32
# workload with its A2 and A5 indices merged into one, so that the 32 rows of
# each 96 x 32 flat tile lie in one plane of A instead of up to 20 planes 13 MB
# apart (same extents, tile shape, bytes and kernel; A(24, 20, 320, 24, 18),
# perm [2, 0, 4, 1, 3]).
#
# And a 2-D fp32 transposition whose 32-element A runs start off the 128-byte
# lines (A rows of 2193 elements), once with the quick plan (tiles dealt to
# the XCDs 16 at a time) and once with the same tiles dealt one by one, round
# robin: neighbouring tiles, which share A's boundary lines, then sit in
# different XCDs' L2s.
DIAGNOSTIC_WORKLOADS = [
    Workload("oneplane6d_24x20x320x24x18_f32", "f32", (24, 20, 320, 24, 18), (2, 0, 4, 1, 3),
             1.5, 0.0, 2, None, knobs=(("run_a", 96), ("run_b", 32))),
    Workload("xcdgroups2d_2193x22800_f32", "f32", (2193, 22800), (1, 0), 1.0, 0.0, 9, None),
    Workload("roundrobin2d_2193x22800_f32", "f32", (2193, 22800), (1, 0), 1.0, 0.0, 9, None,
             knobs=(("xcd_group", 1), ("tile_order", 2))),
]

BY_NAME = {w.name: w for w in WORKLOADS + SUBTENSOR_WORKLOADS + DIAGNOSTIC_WORKLOADS}


def _fortran_offset(index, outer) -> int:
    off, stride = 0, 1
    for i, o in zip(index, outer):
        off += int(i) * stride
        stride *= int(o)
    return off


TORCH_DTYPE = {"f32": torch.float32, "f64": torch.float64}
NUMPY_DTYPE = {"f32": np.float32, "f64": np.float64}


def uniform(numel: int, dtype: str, seed: int) -> torch.Tensor:
    """``numel`` values uniform in [-1, 1) on the CPU, from a seeded generator."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return torch.rand(numel, dtype=TORCH_DTYPE[dtype], generator=g) * 2 - 1


def inputs(w: Workload):
    """Host tensors (A, B_prior) of a workload; B_prior is None when beta == 0."""
    A = uniform(w.numel, w.dtype, w.seed_a)
    B = uniform(w.numel, w.dtype, w.seed_b) if w.seed_b is not None else None
    return A, B


# The paper's benchmark: 57 transpositions of 2-D to 6-D tensors of roughly
# 200 MB each, single precision, reported for beta != 0 unless stated
# (Section 4).  Its case list is not printed; this seeded generator stands in
# for it with the same dimension range, tensor size and precision.
SWEEP_DIMS = {2: 5, 3: 10, 4: 14, 5: 14, 6: 14}      # 57 cases
SWEEP_BYTES = 200 * 1000 * 1000


def sweep57(seed: int = 1704, beta: float = 1.0, alpha: float = 1.0) -> list:
    """57 seeded fp32 workloads, ``SWEEP_BYTES`` per tensor (within 3 %).
    Extents are log-uniform shares of the element count (every extent >= 2,
    so each index is a real one and small leading extents occur); perms are
    uniform over the non-identity permutations, so the stride-1 index is
    kept in about 1/N of the cases."""
    rng = np.random.default_rng(seed)
    target = SWEEP_BYTES // 4
    out = []
    for n, count in SWEEP_DIMS.items():
        for c in range(count):
            while True:
                w = rng.dirichlet(np.ones(n))
                ext = [max(2, int(round(target ** x))) for x in w]
                ext[-1] = max(2, int(round(target / prod(ext[:-1]))))
                if abs(prod(ext) / target - 1) <= 0.03:
                    break
            while True:
                perm = tuple(int(p) for p in rng.permutation(n))
                if perm != tuple(range(n)):
                    break
            name = f"sweep{n}d_{c:02d}_" + "x".join(map(str, ext)) + "_p" + "".join(map(str, perm))
            out.append(Workload(name, "f32", tuple(ext), perm, alpha, beta,
                                seed * 1000 + len(out), None if beta == 0 else seed * 1000 + 500
                                + len(out)))
    return out


@dataclass(frozen=True)
class ContractionWorkload:
    """C[modes_c] = alpha * A[modes_a] . B[modes_b] + beta * C (Fortran order)."""
    name: str
    modes_c: str
    modes_a: str
    modes_b: str
    extents: tuple           # ((mode, extent), ...)
    dtype: str = "f64"
    alpha: float = 1.0
    beta: float = 0.0
    seed: int = 0

    def ext(self) -> dict:
        return dict(self.extents)

    def size(self, modes: str) -> tuple:
        e = self.ext()
        return tuple(e[m] for m in modes)

    def numel(self, modes: str) -> int:
        return prod(self.size(modes))

    @property
    def spec(self) -> str:
        return f"{self.modes_c}={self.modes_a}*{self.modes_b}"

    @property
    def flops(self) -> int:
        e = self.ext()
        return 2 * prod(e[m] for m in set(self.modes_a) | set(self.modes_b))


def _cw(name, spec, dtype="f64", **ext):
    c, ab = spec.split("=")
    a, b = ab.split("*")
    return ContractionWorkload(name, c, a, b, tuple(sorted(ext.items())), dtype)


# Contractions standing in for the tensor-contraction experiment of Section
# 4.1 (double precision, like Fig. 9), whose case list is not in the paper:
# from bandwidth-bound (few contracted elements, large C) to compute-bound
# (long contractions), plus a pure matrix product that needs no transposition.
CONTRACTIONS = [
    _cw("abcd_aebf_dfce", "abcd=aebf*dfce", a=72, b=72, c=72, d=72, e=4, f=4),
    _cw("abcd_ebad_ce", "abcd=ebad*ce", a=48, b=48, c=256, d=48, e=16),
    _cw("abc_bda_dc", "abc=bda*dc", a=512, b=256, c=256, d=24),
    _cw("abcde_efbad_cf", "abcde=efbad*cf", a=24, b=24, c=96, d=24, e=24, f=32),
    _cw("abcd_dbea_ec", "abcd=dbea*ec", a=96, b=64, c=96, d=64, e=64),
    _cw("ab_acd_dbc", "ab=acd*dbc", a=2048, b=2048, c=64, d=64),
    _cw("abc_adec_ebd", "abc=adec*ebd", a=96, b=96, c=96, d=96, e=96),
    _cw("ij_ik_kj", "ij=ik*kj", i=4096, j=4096, k=4096),
]
CONTRACTIONS_BY_NAME = {w.name: w for w in CONTRACTIONS}


def random_problem(rng: np.random.Generator, max_dims: int = 6,
                   extents=(1, 2, 3, 5, 7, 17, 33, 64, 65), max_numel: int = 1 << 20):
    """A random (size_a, perm) pair for sweeps, with at most ``max_numel`` elements."""
    while True:
        n = int(rng.integers(1, max_dims + 1))
        size_a = tuple(int(rng.choice(extents)) for _ in range(n))
        if prod(size_a) <= max_numel:
            perm = tuple(int(p) for p in rng.permutation(n))
            return size_a, perm
