"""Pins of the CPU oracle against what the paper and mathematics fix (CPU only).

Each ``pin_*`` function takes an oracle library and raises AssertionError when
it disagrees with something other than itself: a worked example printed in
the paper (fixtures under tests/golden/, each with its citation), numpy's
transpose, exact rational arithmetic, a pure-Python brute force, or an
invariant of Eq. (1).  The same battery is then run against deliberately
broken copies of the oracle (``test_pins_catch_planted_mistakes``) to show that
a plausible mistake anywhere in it fails at least one pin.
"""
from __future__ import annotations

import itertools
import os
import shutil
import subprocess
import sys
from fractions import Fraction

import numpy as np
import pytest

from conftest import ROOT, golden
from oracle import brute
from oracle import oracle as oracle_mod

RNG_SEED = 20170414


def _rand(rng, n, dtype):
    # Values in [-1, 1) on a 2^-20 grid: exact in both dtypes, never subnormal.
    return (rng.integers(-(1 << 20), 1 << 20, size=n) / float(1 << 20)).astype(dtype)


def _numpy_transpose(A, size_a, perm):
    """numpy.transpose on the Fortran view: axis k of the result is axis
    perm[k] of A, which is exactly the convention B dim k = A dim perm[k]."""
    return np.transpose(A.reshape(size_a, order="F"), perm).ravel(order="F")


def _inverse(perm):
    inv = [0] * len(perm)
    for k, p in enumerate(perm):
        inv[p] = k
    return tuple(inv)


# --------------------------------------------------------------------------
# Pins from the paper's worked examples
# --------------------------------------------------------------------------

def pin_fig1_strides(orc):
    """Fig. 1: in B_{i2 i1} <- A_{i1 i2} with A 6x4, index i1 has strides 1
    (A) and 4 (B) over 0..5; i2 has strides 6 (A) and 1 (B) over 0..3."""
    rows = {r[0]: r[1:] for r in golden("fig1_plan.txt")}
    size_a = tuple(int(x) for x in rows["sizeA"])
    perm = tuple(int(x) for x in rows["perm"])
    i1 = [int(x) for x in rows["i1"]]
    i2 = [int(x) for x in rows["i2"]]
    A = np.arange(24, dtype=np.float32)
    B = orc.transpose(A, size_a, perm)
    assert orc.size_b(size_a, perm) == (4, 6)
    for a in range(i1[0], i1[1], i1[2]):
        for b in range(i2[0], i2[1], i2[2]):
            assert B[a * i1[4] + b * i2[4]] == A[a * i1[3] + b * i2[3]]


def pin_fig3b_sizes(orc):
    """Fig. 3b: perm {2,1,0} on sizeA {8,16,16} gives the compact B
    16x16x8 (its outer size), and B_{i3 i2 i1} = A_{i1 i2 i3}."""
    rows = {r[0]: r[1:] for r in golden("fig3b_input.txt")}
    perm = tuple(int(x) for x in rows["perm"])
    size_a = tuple(int(x) for x in rows["sizeA"])
    size_b = tuple(int(x) for x in rows["outerSizeB"])
    assert orc.size_b(size_a, perm) == size_b
    A = np.arange(int(np.prod(size_a)), dtype=np.float32)
    B = orc.transpose(A, size_a, perm, float(rows["alpha"][0]), float(rows["beta"][0]))
    Af = A.reshape(size_a, order="F")
    Bf = B.reshape(size_b, order="F")
    for i1, i2, i3 in itertools.product(*[range(n) for n in size_a]):
        assert Bf[i3, i2, i1] == Af[i1, i2, i3]


def pin_fn4_fusion(orc):
    """Footnote 4: B_{i2 i3 i1} <- A_{i1 i2 i3} is B_{(i2 i3) i1} <- A_{i1 (i2 i3)}."""
    rows = {r[0]: r[1:] for r in golden("fn4_fusion.txt")}
    perm = tuple(int(x) for x in rows["perm"])
    fused = tuple(int(x) for x in rows["fused_perm"])
    rng = np.random.default_rng(RNG_SEED)
    for n1, n2, n3 in [(3, 4, 5), (7, 2, 6), (1, 5, 3), (4, 1, 2)]:
        for dtype, alpha, beta in [(np.float32, 1.0, 0.0), (np.float64, -0.75, 1.25)]:
            A = _rand(rng, n1 * n2 * n3, dtype)
            B0 = _rand(rng, n1 * n2 * n3, dtype)
            full = orc.transpose(A, (n1, n2, n3), perm, alpha, beta, B0)
            merged = orc.transpose(A, (n1, n2 * n3), fused, alpha, beta, B0)
            assert np.array_equal(full, merged)


def pin_table1_notation(orc):
    """Table 1 and its text: the column "6,1,5,4,3,2" is B_{i6 i1 i5 i4 i3 i2},
    i.e. B's fastest index is A's i6 and its second fastest is A's i1."""
    size_a = (2, 3, 4, 5, 6, 7)          # distinct extents expose a swapped reading
    strides_a = np.cumprod((1,) + size_a[:-1])
    for label, order, fastest, second in golden("table1.txt"):
        perm = tuple(int(x) - 1 for x in order.split(","))
        f, s = int(fastest) - 1, int(second) - 1
        assert perm[0] == f and perm[1] == s, label
        size_b = orc.size_b(size_a, perm)
        assert size_b[0] == size_a[f] and size_b[1] == size_a[s], label
        A = np.arange(int(np.prod(size_a)), dtype=np.float64)
        B = orc.transpose(A, size_a, perm)
        # walking B's first index walks A's index f; B's second walks A's s
        assert np.array_equal(B[:size_b[0]], np.arange(size_b[0]) * strides_a[f]), label
        assert np.array_equal(B[0:size_b[0] * size_b[1]:size_b[0]],
                              np.arange(size_b[1]) * strides_a[s]), label


# --------------------------------------------------------------------------
# Pins from library routines and textbook special cases
# --------------------------------------------------------------------------

def pin_numpy_transpose(orc):
    """A random sweep against numpy.transpose (alpha=1, beta=0, bit-exact) and
    against numpy's per-operation rounded arithmetic for general alpha, beta."""
    rng = np.random.default_rng(RNG_SEED + 1)
    for _ in range(60):
        n = int(rng.integers(1, 7))
        size_a = tuple(int(x) for x in rng.choice([1, 2, 3, 4, 5, 7], size=n))
        perm = tuple(int(p) for p in rng.permutation(n))
        for dtype in (np.float32, np.float64):
            A = _rand(rng, int(np.prod(size_a)), dtype)
            B0 = _rand(rng, A.size, dtype)
            ref = _numpy_transpose(A, size_a, perm)
            assert np.array_equal(orc.transpose(A, size_a, perm), ref)
            alpha, beta = dtype(rng.uniform(-2, 2)), dtype(rng.uniform(-2, 2))
            expect = alpha * ref + beta * B0       # each numpy op rounds once
            got = orc.transpose(A, size_a, perm, float(alpha), float(beta), B0)
            assert np.array_equal(got, expect)
            got0 = orc.transpose(A, size_a, perm, float(alpha), 0.0)
            assert np.array_equal(got0, alpha * ref)


def pin_identity_is_axpby(orc):
    """The identity permutation reduces Eq. (1) to B <- alpha*A + beta*B, the
    SAXPY-like operation of Table 2."""
    rng = np.random.default_rng(RNG_SEED + 2)
    for size_a in [(1000,), (5, 7), (3, 4, 5), (2, 3, 1, 4)]:
        perm = tuple(range(len(size_a)))
        for dtype in (np.float32, np.float64):
            A = _rand(rng, int(np.prod(size_a)), dtype)
            B0 = _rand(rng, A.size, dtype)
            alpha, beta = dtype(1.5), dtype(-0.375)
            got = orc.transpose(A, size_a, perm, float(alpha), float(beta), B0)
            assert np.array_equal(got, alpha * A + beta * B0)


def pin_matrix_transpose(orc):
    """N = 2 with perm (1, 0) is the matrix transpose of Section 2."""
    rng = np.random.default_rng(RNG_SEED + 3)
    for n1, n2 in [(6, 4), (1, 9), (33, 17), (64, 65)]:
        A = _rand(rng, n1 * n2, np.float32)
        B = orc.transpose(A, (n1, n2), (1, 0))
        assert np.array_equal(B.reshape((n2, n1), order="F"), A.reshape((n1, n2), order="F").T)


def pin_brute_force(orc):
    """Every permutation of rank <= 4 on small extents against the
    independent pure-Python brute force of the definition."""
    rng = np.random.default_rng(RNG_SEED + 4)
    cases = [(1.0, 0.0), (1.5, 0.0), (-0.3, 1.25), (2.0, 0.5)]
    for n in range(1, 5):
        for perm in itertools.permutations(range(n)):
            size_a = tuple(int(x) for x in rng.choice([1, 2, 3, 5], size=n))
            for dtype in (np.float32, np.float64):
                A = _rand(rng, int(np.prod(size_a)), dtype)
                B0 = _rand(rng, A.size, dtype)
                alpha, beta = cases[int(rng.integers(len(cases)))]
                want = np.array(brute.transpose(list(A), size_a, perm, alpha, beta,
                                                list(B0), dtype), dtype=dtype)
                got = orc.transpose(A, size_a, perm, alpha, beta, B0)
                assert np.array_equal(got, want), (perm, size_a, dtype, alpha, beta)


def _round_to(dtype, q: Fraction):
    # float(Fraction) is correctly rounded to double; the fp32 cases are built
    # so that q is exact in double, making the second rounding the only one.
    x = float(q)
    if dtype == np.float32:
        assert Fraction(x) == q
        return np.float32(x)
    return np.float64(x)


def pin_two_roundings(orc):
    """Reading of the rounding: fl(fl(alpha*a) + fl(beta*b)) in the tensor
    dtype, never a fused multiply-add.  Checked with exact rational arithmetic
    on inputs where the fused result would differ."""
    rng = np.random.default_rng(RNG_SEED + 5)
    for dtype in (np.float32, np.float64):
        found = 0
        while found < 8:
            alpha, beta = dtype(rng.uniform(0.5, 2)), dtype(rng.uniform(0.5, 2))
            a, b = dtype(rng.uniform(-1, 1)), dtype(rng.uniform(-1, 1))
            pa = _round_to(dtype, Fraction(float(alpha)) * Fraction(float(a)))
            pb = _round_to(dtype, Fraction(float(beta)) * Fraction(float(b)))
            two = _round_to(dtype, Fraction(float(pa)) + Fraction(float(pb)))
            fused = _round_to(dtype, Fraction(float(alpha)) * Fraction(float(a))
                              + Fraction(float(pb))) if dtype == np.float64 else \
                np.float32(float(Fraction(float(alpha)) * Fraction(float(a)) + Fraction(float(pb))))
            if two == fused:
                continue
            found += 1
            A = np.array([a, a], dtype=dtype)
            B0 = np.array([b, b], dtype=dtype)
            got = orc.transpose(A, (2,), (0,), float(alpha), float(beta), B0)
            assert got[0] == two and got[1] == two, (dtype, alpha, beta, a, b)


# --------------------------------------------------------------------------
# Pins from invariants of Eq. (1)
# --------------------------------------------------------------------------

def pin_inverse_roundtrip(orc):
    """Applying Pi and then Pi^-1 returns A bit for bit."""
    rng = np.random.default_rng(RNG_SEED + 6)
    for _ in range(20):
        n = int(rng.integers(1, 7))
        size_a = tuple(int(x) for x in rng.choice([1, 2, 3, 5, 6], size=n))
        perm = tuple(int(p) for p in rng.permutation(n))
        A = _rand(rng, int(np.prod(size_a)), np.float64)
        B = orc.transpose(A, size_a, perm)
        back = orc.transpose(B, orc.size_b(size_a, perm), _inverse(perm))
        assert np.array_equal(back, A)


def pin_hit_once(orc):
    """Every B element is written exactly once: with A = 1, B = 0 and
    alpha = beta = 1 every element becomes 1, and with A holding its own
    offsets B holds a permutation of 0..numel-1."""
    for size_a, perm in [((3, 4, 5), (2, 0, 1)), ((2, 3, 2, 5), (1, 3, 0, 2)),
                         ((7, 1, 6), (0, 2, 1))]:
        numel = int(np.prod(size_a))
        ones = orc.transpose(np.ones(numel, np.float32), size_a, perm, 1.0, 1.0,
                             np.zeros(numel, np.float32))
        assert np.all(ones == 1)
        idx = orc.transpose(np.arange(numel, dtype=np.float32), size_a, perm)
        assert np.array_equal(np.sort(idx), np.arange(numel, dtype=np.float32))


def pin_beta_zero_does_not_read_b(orc):
    """Reading of Eq. (2)'s lambda = 2: with beta = 0 B is only written, so a
    NaN or inf already in B never reaches the result."""
    rng = np.random.default_rng(RNG_SEED + 7)
    size_a, perm = (5, 6, 7), (2, 1, 0)
    for dtype in (np.float32, np.float64):
        A = _rand(rng, 210, dtype)
        B0 = np.full(210, np.nan, dtype=dtype)
        B0[::3] = np.inf
        for alpha in (1.0, -2.5):
            got = orc.transpose(A, size_a, perm, alpha, 0.0, B0)
            assert not np.any(np.isnan(got)) and not np.any(np.isinf(got))
            assert np.array_equal(got, dtype(alpha) * _numpy_transpose(A, size_a, perm))


def pin_alpha_zero_still_reads_a(orc):
    """Reading of footnote 5: alpha = 0 is not short-cut, A is still read and
    multiplied, so an inf in A turns into NaN in B."""
    size_a, perm = (4, 3), (1, 0)
    A = np.ones(12, dtype=np.float32)
    A[5] = np.inf                      # A index (1, 1) -> B offset 1 + 3*1 = 4
    B0 = np.full(12, 0.25, dtype=np.float32)
    got = orc.transpose(A, size_a, perm, 0.0, 1.0, B0)
    assert np.isnan(got[4])
    assert np.all(np.delete(got, 4) == 0.25)


def pin_sample_matches_full(orc):
    """The one-by-one sampler agrees with the whole transposition."""
    rng = np.random.default_rng(RNG_SEED + 8)
    size_a, perm = (5, 4, 3, 6), (3, 1, 0, 2)
    A = _rand(rng, 360, np.float64)
    B0 = _rand(rng, 360, np.float64)
    full = orc.transpose(A, size_a, perm, 1.5, -0.5, B0)
    offs = rng.integers(0, 360, size=50)
    assert np.array_equal(orc.sample(A, size_a, perm, 1.5, -0.5, B0, offs), full[offs])


# --------------------------------------------------------------------------
# Pins of sub-tensors with outer sizes (Section 3.1, Fig. 3)
# --------------------------------------------------------------------------

def _fortran_offset(index, outer):
    off, stride = 0, 1
    for i, o in zip(index, outer):
        off += int(i) * stride
        stride *= int(o)
    return off


def pin_fig3b_outer_sizes(orc):
    """Fig. 3: the 8x16x16 sub-tensor of A (outer 16x32x32) transposed and
    compacted into B (outer = size = 16x16x8), against numpy slicing."""
    rows = {r[0]: r[1:] for r in golden("fig3b_input.txt")}
    perm = tuple(int(x) for x in rows["perm"])
    size_a = tuple(int(x) for x in rows["sizeA"])
    outer_a = tuple(int(x) for x in rows["outerSizeA"])
    outer_b = tuple(int(x) for x in rows["outerSizeB"])
    A = np.arange(int(np.prod(outer_a)), dtype=np.float32)
    B = orc.transpose_outer(A, size_a, perm, outer_a, outer_b)
    sub = A.reshape(outer_a, order="F")[tuple(slice(0, n) for n in size_a)]
    assert np.array_equal(B, np.transpose(sub, perm).ravel(order="F"))


def pin_outer_sizes_numpy(orc):
    """Random sub-tensors at random positions of larger tensors, compacted
    and scattered: the sub-tensor of B equals numpy's transpose of the
    sub-tensor of A, and every other element of B keeps its value."""
    rng = np.random.default_rng(RNG_SEED + 9)
    for it in range(40):
        n = int(rng.integers(1, 5))
        size_a = tuple(int(x) for x in rng.integers(1, 5, size=n))
        perm = tuple(int(p) for p in rng.permutation(n))
        size_b = tuple(size_a[p] for p in perm)
        outer_a = tuple(s + int(rng.integers(0, 3)) for s in size_a)
        outer_b = tuple(s + int(rng.integers(0, 3)) for s in size_b)
        start_a = tuple(int(rng.integers(0, o - s + 1)) for s, o in zip(size_a, outer_a))
        start_b = tuple(int(rng.integers(0, o - s + 1)) for s, o in zip(size_b, outer_b))
        dtype = (np.float32, np.float64)[it % 2]
        alpha, beta = ((1.0, 0.0), (1.5, -0.5), (-2.0, 0.25))[it % 3]
        PA = _rand(rng, int(np.prod(outer_a)), dtype)
        PB = _rand(rng, int(np.prod(outer_b)), dtype)
        oa, ob = _fortran_offset(start_a, outer_a), _fortran_offset(start_b, outer_b)
        got_tail = orc.transpose_outer(PA[oa:], size_a, perm, outer_a, outer_b, alpha, beta,
                                       PB[ob:])
        got = np.concatenate([PB[:ob], got_tail])
        sl_a = tuple(slice(s, s + n) for s, n in zip(start_a, size_a))
        sl_b = tuple(slice(s, s + n) for s, n in zip(start_b, size_b))
        want = PB.reshape(outer_b, order="F").copy()
        t = np.transpose(PA.reshape(outer_a, order="F")[sl_a], perm)
        want[sl_b] = dtype(alpha) * t + dtype(beta) * want[sl_b] if beta != 0 else dtype(alpha) * t
        assert np.array_equal(got, want.ravel(order="F")), (size_a, perm, outer_a, outer_b)


def pin_outer_equal_to_size_is_compact(orc):
    """Outer sizes equal to the sizes give the compact transposition."""
    rng = np.random.default_rng(RNG_SEED + 10)
    for size_a, perm in [((3, 4, 5), (2, 0, 1)), ((6, 7), (1, 0)), ((2, 3, 2, 5), (3, 1, 0, 2))]:
        A = _rand(rng, int(np.prod(size_a)), np.float64)
        B0 = _rand(rng, A.size, np.float64)
        size_b = tuple(size_a[p] for p in perm)
        assert np.array_equal(orc.transpose_outer(A, size_a, perm, size_a, size_b, 1.5, 0.5, B0),
                              orc.transpose(A, size_a, perm, 1.5, 0.5, B0))


PINS = [pin_fig1_strides, pin_fig3b_sizes, pin_fn4_fusion, pin_table1_notation,
        pin_numpy_transpose, pin_identity_is_axpby, pin_matrix_transpose, pin_brute_force,
        pin_two_roundings, pin_inverse_roundtrip, pin_hit_once,
        pin_beta_zero_does_not_read_b, pin_alpha_zero_still_reads_a, pin_sample_matches_full,
        pin_fig3b_outer_sizes, pin_outer_sizes_numpy, pin_outer_equal_to_size_is_compact]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin, oracle_lib):
    pin(oracle_lib)


def test_invalid_problems_rejected(oracle_lib):
    with pytest.raises(ValueError):
        oracle_lib.size_b((2, 3), (0, 0))
    with pytest.raises(ValueError):
        oracle_lib.size_b((2, 3), (0, 2))
    with pytest.raises(ValueError):
        oracle_lib.size_b((2, -1), (1, 0))


def test_zero_extent_is_noop(oracle_lib):
    A = np.zeros(0, dtype=np.float32)
    B = oracle_lib.transpose(A, (4, 0, 3), (2, 1, 0))
    assert B.size == 0


# --------------------------------------------------------------------------
# Planted mistakes: each must fail at least one pin
# --------------------------------------------------------------------------

MUTANTS = {
    "dropped_beta_term": [("return scaled_a + scaled_b;", "return scaled_a;")],
    "wrong_sign": [("return scaled_a + scaled_b;", "return scaled_a - scaled_b;")],
    "alpha_ignored": [("return alpha * a;", "return a;")],
    "b_read_when_beta_zero": [("if (beta == 0.0f) {", "if (0) {"), ("if (beta == 0.0) {", "if (0) {"),
                              ("beta == 0.0f ? 0.0f : B[offB]", "B[offB]"),
                              ("beta == 0.0 ? 0.0 : B[offB]", "B[offB]")],
    "fused_multiply_add": [("return scaled_a + scaled_b;", "return fmaf(alpha, a, scaled_b);"),
                           ("#include <stdint.h>", "#include <stdint.h>\n#include <math.h>")],
    "perm_direction_inverted": [("b += i[perm[k]] * strideB[k];", "b += i[k] * strideB[perm[k]];")],
    "size_b_inverted": [("for (int k = 0; k < N; ++k) sizeB[k] = sizeA[perm[k]];",
                         "for (int k = 0; k < N; ++k) sizeB[perm[k]] = sizeA[k];")],
    "b_strides_from_a_sizes": [("fortran_strides(N, outerB, strideB);",
                                "fortran_strides(N, outerA, strideB);")],
    "outer_a_ignored": [("outerA[d] = outerSizeA ? outerSizeA[d] : sizeA[d];",
                         "outerA[d] = sizeA[d];")],
    "outer_b_in_a_order": [("outerB[d] = outerSizeB ? outerSizeB[d] : sizeB[d];",
                            "outerB[d] = outerSizeB ? outerSizeB[perm[d]] : sizeB[d];")],
    "a_offset_uses_b_strides": [("for (int d = 0; d < N; ++d) a += i[d] * strideA[d];\n    for (int k",
                                 "for (int d = 0; d < N; ++d) a += i[d] * strideB[d];\n    for (int k")],
    "stride_off_by_one": [("stride[d] = stride[d - 1] * size[d - 1];",
                           "stride[d] = stride[d - 1] * size[d];")],
    "alpha_beta_swapped": [("float scaled_a = alpha * a;", "float scaled_a = beta * a;"),
                           ("float scaled_b = beta * b;", "float scaled_b = alpha * b;")],
    "copy_when_alpha_not_one": [("if (alpha == 1.0) return a;", "return a;")],
}


_MUTANT_RUNNER = """
import sys
sys.path.insert(0, {tests!r})
sys.path.insert(0, {root!r})
import test_oracle as t
from oracle import oracle as om
m = om.OracleLib({lib!r})
for pin in t.PINS:
    print("RUN", pin.__name__, flush=True)
    try:
        pin(m)
    except (AssertionError, ValueError):
        print("FAIL", pin.__name__, flush=True)
"""


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistakes(name, tmp_path):
    """A broken oracle may index out of bounds, so each one runs in a child
    process; a crash inside a pin counts as that pin catching the mistake."""
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    for old, new in MUTANTS[name]:
        assert old in src, f"mutation anchor missing: {old!r}"
        src = src.replace(old, new)
    path = tmp_path / "mutant.c"
    path.write_text(src)
    lib = oracle_mod.compile_source(str(path), str(tmp_path / "libmutant.so"))
    code = _MUTANT_RUNNER.format(tests=os.path.join(ROOT, "tests"), root=ROOT, lib=lib)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       timeout=300)
    lines = r.stdout.splitlines()
    caught = [ln.split()[1] for ln in lines if ln.startswith("FAIL")]
    if r.returncode != 0:
        ran = [ln.split()[1] for ln in lines if ln.startswith("RUN")]
        assert ran, r.stderr[-2000:]
        caught.append(ran[-1] + " (crashed)")
    assert caught, f"no pin catches the planted mistake {name}"
    shutil.rmtree(tmp_path, ignore_errors=True)
