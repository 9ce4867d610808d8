"""Oracle for a tensor contraction, the operation the paper's transpositions
serve inside a tensor-contraction framework (Sections 1 and 4.1: a
contraction cast as transpositions around a matrix-matrix product):

    C_{modesC}  <-  alpha * sum over the contracted modes of A_{modesA} * B_{modesB}
                    +  beta * C_{modesC}

All tensors are in the Fortran layout of Section 1 (first mode fastest).
Modes are single letters; a mode of C appears in A or B (or both: a batch
mode), a mode in A and B but not C is summed over.  Each mode appears at
most once per tensor.

TEST INFRASTRUCTURE, NOT PRODUCT CODE: only the test-suite and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the GPU library.  The sum is numpy's einsum in float64 (a library primitive
that evaluates the definition above), whatever the input dtype.
"""
from __future__ import annotations

import numpy as np


def _check(modes: str, size, what: str):
    if len(set(modes)) != len(modes):
        raise ValueError(f"{what}: a mode repeats in {modes!r}")
    if len(size) != len(modes):
        raise ValueError(f"{what}: {len(modes)} modes but {len(size)} extents")


def extents(modes_a: str, size_a, modes_b: str, size_b) -> dict:
    """The extent of every mode of A and B (equal where they share one)."""
    ext = {}
    for modes, size in ((modes_a, size_a), (modes_b, size_b)):
        for m, s in zip(modes, size):
            if ext.setdefault(m, int(s)) != int(s):
                raise ValueError(f"mode {m!r} has extents {ext[m]} and {s}")
    return ext


def _tensor(x: np.ndarray, size) -> np.ndarray:
    """A flat Fortran-ordered array as an n-d float64 view."""
    return np.asarray(x, dtype=np.float64).reshape(tuple(int(s) for s in size), order="F")


def contract(A: np.ndarray, modes_a: str, size_a, B: np.ndarray, modes_b: str, size_b,
             modes_c: str, alpha: float = 1.0, beta: float = 0.0,
             C: np.ndarray | None = None) -> np.ndarray:
    """C as a flat float64 Fortran-ordered array."""
    _check(modes_a, size_a, "A")
    _check(modes_b, size_b, "B")
    ext = extents(modes_a, size_a, modes_b, size_b)
    if len(set(modes_c)) != len(modes_c) or any(m not in ext for m in modes_c):
        raise ValueError(f"C modes {modes_c!r} must be distinct modes of A or B")
    for m in modes_a:
        if m not in modes_b and m not in modes_c:
            raise ValueError(f"mode {m!r} of A is neither in B nor in C")
    for m in modes_b:
        if m not in modes_a and m not in modes_c:
            raise ValueError(f"mode {m!r} of B is neither in A nor in C")
    size_c = [ext[m] for m in modes_c]
    prod = np.einsum(f"{modes_a},{modes_b}->{modes_c}", _tensor(A, size_a), _tensor(B, size_b),
                     optimize=False)
    out = float(alpha) * prod
    if beta != 0:
        if C is None:
            raise ValueError("beta != 0 needs the prior C")
        out = out + float(beta) * _tensor(C, size_c)
    return np.asarray(out).reshape(-1, order="F")


def contract_sample(A: np.ndarray, modes_a: str, size_a, B: np.ndarray, modes_b: str, size_b,
                    modes_c: str, offsets_c, alpha: float = 1.0, beta: float = 0.0,
                    C: np.ndarray | None = None):
    """(value, magnitude) of C at the given Fortran offsets of C, each
    computed on its own from the definition: split the offset into C's
    mode indices, fix those modes in A and B, and sum the products over the
    contracted modes (for tensors too large to contract whole on the CPU)."""
    ext = extents(modes_a, size_a, modes_b, size_b)
    size_c = [ext[m] for m in modes_c]
    ta, tb = _tensor(A, size_a), _tensor(B, size_b)
    con = "".join(m for m in modes_a if m in modes_b and m not in modes_c)
    vals, mags = [], []
    for off in np.asarray(offsets_c, dtype=np.int64):
        idx, rest = {}, int(off)
        for m, n in zip(modes_c, size_c):
            idx[m] = rest % n
            rest //= n
        sa = tuple(idx.get(m, slice(None)) for m in modes_a)
        sb = tuple(idx.get(m, slice(None)) for m in modes_b)
        ra = "".join(m for m in modes_a if m not in idx)
        rb = "".join(m for m in modes_b if m not in idx)
        xa, xb = ta[sa], tb[sb]
        dot = float(np.einsum(f"{ra},{rb}->", xa, xb, optimize=False)) if con else float(xa * xb)
        mag = (float(np.einsum(f"{ra},{rb}->", np.abs(xa), np.abs(xb), optimize=False)) if con
               else float(abs(xa * xb)))
        v, g = float(alpha) * dot, abs(float(alpha)) * mag
        if beta != 0:
            c0 = float(np.asarray(C, dtype=np.float64)[off])
            v += float(beta) * c0
            g += abs(float(beta)) * abs(c0)
        vals.append(v)
        mags.append(g)
    return np.array(vals), np.array(mags)


def magnitude(A: np.ndarray, modes_a: str, size_a, B: np.ndarray, modes_b: str, size_b,
              modes_c: str, alpha: float = 1.0, beta: float = 0.0,
              C: np.ndarray | None = None) -> np.ndarray:
    """|alpha| * sum |A| |B| + |beta| |C|: the scale of the rounding error a
    summation of the products in any order may make (flat, Fortran order)."""
    return contract(np.abs(np.asarray(A, dtype=np.float64)), modes_a, size_a,
                    np.abs(np.asarray(B, dtype=np.float64)), modes_b, size_b, modes_c,
                    abs(alpha), abs(beta),
                    None if C is None else np.abs(np.asarray(C, dtype=np.float64)))


def error_bound(mag: np.ndarray, k: int, dtype: str) -> np.ndarray:
    """Elementwise bound on |computed - exact| for a dot product of length k
    summed in any order in the given precision, plus the roundings of the
    alpha and beta products and of the final sum: (k + 2) * u * mag
    (Higham, Accuracy and Stability of Numerical Algorithms, Section 3.1,
    gamma_n = n u / (1 - n u), first order)."""
    u = 2.0 ** -24 if dtype == "f32" else 2.0 ** -53
    return (k + 2) * u * mag * (1 + 1e-6)
