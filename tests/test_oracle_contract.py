"""Pins of the contraction oracle (oracle/contract.py) against what the
mathematics fixes independently of it: brute-force sums on tiny shapes, the
matrix product, the outer product, batched matrix products, a contraction
with the identity matrix that is a transposition (checked against the
transposition oracle), linearity in alpha and beta, and the error bound's
reach.  Planted mistakes in a copy of the oracle must fail them."""
from __future__ import annotations

import itertools

import numpy as np
import pytest

from oracle import contract as oc
from oracle import oracle as orc


def _rand(rng, n):
    return rng.integers(-8, 8, size=n).astype(np.float64) / 8.0


def _brute(A, ma, sa, B, mb, sb, mc, alpha, beta, C):
    """Every output index, every contracted index, in plain loops over
    Fortran offsets."""
    ext = dict(zip(ma, sa))
    ext.update(zip(mb, sb))
    con = [m for m in ext if m not in mc]
    sc = [ext[m] for m in mc]

    def off(modes, idx):
        o, s = 0, 1
        for m in modes:
            o += idx[m] * s
            s *= ext[m]
        return o

    out = np.zeros(int(np.prod(sc)) if sc else 1)
    for cidx in itertools.product(*[range(ext[m]) for m in mc]):
        idx = dict(zip(mc, cidx))
        acc = 0.0
        for kidx in itertools.product(*[range(ext[m]) for m in con]):
            idx.update(zip(con, kidx))
            acc += A[off(ma, idx)] * B[off(mb, idx)]
        o = off(mc, idx)
        out[o] = alpha * acc + (beta * C[o] if beta else 0.0)
    return out


CASES = [
    ("ab", (3, 4), "bc", (4, 5), "ac"),
    ("abc", (2, 3, 4), "cbd", (4, 3, 5), "da"),
    ("aebf", (2, 3, 2, 2), "dfce", (3, 2, 2, 3), "abcd"),
    ("akl", (3, 4, 2), "kbl", (4, 5, 2), "abl"),          # batch mode l
    ("a", (4,), "b", (3,), "ba"),                         # outer product
    ("kab", (5, 2, 3), "kc", (5, 2), "cba"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}*{c[2]}->{c[4]}")
def test_brute_force(case):
    ma, sa, mb, sb, mc = case
    rng = np.random.default_rng(len(ma) * 7 + len(mb))
    A, B = _rand(rng, int(np.prod(sa))), _rand(rng, int(np.prod(sb)))
    ext = oc.extents(ma, sa, mb, sb)
    C = _rand(rng, int(np.prod([ext[m] for m in mc])))
    for alpha, beta in ((1.0, 0.0), (-1.5, 0.75)):
        got = oc.contract(A, ma, sa, B, mb, sb, mc, alpha, beta, C)
        want = _brute(A, ma, sa, B, mb, sb, mc, alpha, beta, C)
        assert np.array_equal(got, want)     # small dyadic values: every sum exact


def test_matrix_product():
    rng = np.random.default_rng(1)
    m, k, n = 7, 5, 6
    A, B = rng.standard_normal(m * k), rng.standard_normal(k * n)
    got = oc.contract(A, "ik", (m, k), B, "kj", (k, n), "ij")
    want = (A.reshape(m, k, order="F") @ B.reshape(k, n, order="F")).reshape(-1, order="F")
    np.testing.assert_allclose(got, want, rtol=1e-14, atol=1e-14)
    # C^T = B^T A^T: the same numbers with the output modes swapped
    got_t = oc.contract(A, "ik", (m, k), B, "kj", (k, n), "ji")
    np.testing.assert_allclose(got_t, want.reshape(m, n, order="F").T.reshape(-1, order="F"),
                               rtol=1e-14, atol=1e-14)


def test_batched_products():
    rng = np.random.default_rng(2)
    m, k, n, l = 4, 3, 5, 6
    A, B = rng.standard_normal(m * k * l), rng.standard_normal(k * n * l)
    got = oc.contract(A, "ikl", (m, k, l), B, "kjl", (k, n, l), "ijl").reshape(
        (m, n, l), order="F")
    a, b = A.reshape(m, k, l, order="F"), B.reshape(k, n, l, order="F")
    for x in range(l):
        np.testing.assert_allclose(got[:, :, x], a[:, :, x] @ b[:, :, x], rtol=1e-13,
                                   atol=1e-14)


def test_identity_contraction_is_a_transposition():
    """C_{c b a} = A_{a k c} delta_{k b}: Eq. (1) with perm (2, 1, 0) once k
    is renamed b -- checked against the transposition oracle."""
    rng = np.random.default_rng(3)
    sa = (4, 3, 5)
    A = rng.standard_normal(int(np.prod(sa)))
    eye = np.eye(3).reshape(-1, order="F")
    got = oc.contract(A, "akc", sa, eye, "kb", (3, 3), "cba")
    want = orc.transpose(A, sa, (2, 1, 0), 1.0, 0.0, None)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}*{c[2]}->{c[4]}")
def test_sample_agrees_with_whole_contraction(case):
    """The one-element-at-a-time definition against the whole-tensor one."""
    ma, sa, mb, sb, mc = case
    rng = np.random.default_rng(11)
    A, B = _rand(rng, int(np.prod(sa))), _rand(rng, int(np.prod(sb)))
    ext = oc.extents(ma, sa, mb, sb)
    nc = int(np.prod([ext[m] for m in mc]))
    C = _rand(rng, nc)
    whole = oc.contract(A, ma, sa, B, mb, sb, mc, -1.25, 0.5, C)
    mag = oc.magnitude(A, ma, sa, B, mb, sb, mc, -1.25, 0.5, C)
    offs = np.arange(nc)
    vals, mags = oc.contract_sample(A, ma, sa, B, mb, sb, mc, offs, -1.25, 0.5, C)
    assert np.array_equal(vals, whole) and np.array_equal(mags, mag)


def test_linearity_in_alpha_and_beta():
    rng = np.random.default_rng(4)
    sa, sb = (3, 4, 2), (4, 5)
    A, B = _rand(rng, 24), _rand(rng, 20)
    C = _rand(rng, 30)
    ab = oc.contract(A, "akb", sa, B, "kc", sb, "abc")
    got = oc.contract(A, "akb", sa, B, "kc", sb, "abc", 2.0, -0.5, C)
    assert np.array_equal(got, 2.0 * ab - 0.5 * C)


def test_invalid_problems():
    with pytest.raises(ValueError):
        oc.contract(np.zeros(4), "aa", (2, 2), np.zeros(2), "b", (2,), "ab")
    with pytest.raises(ValueError):
        oc.contract(np.zeros(4), "ab", (2, 2), np.zeros(3), "b", (3,), "a")
    with pytest.raises(ValueError):
        oc.contract(np.zeros(4), "ab", (2, 2), np.zeros(2), "c", (2,), "ac")  # b summed alone
    with pytest.raises(ValueError):
        oc.contract(np.zeros(4), "ab", (2, 2), np.zeros(2), "b", (2,), "a", 1.0, 1.0)


def test_error_bound_covers_float32_sums():
    """A float32 dot product summed in a bad order stays inside the bound."""
    rng = np.random.default_rng(5)
    k = 4096
    A = rng.standard_normal(k).astype(np.float32)
    B = rng.standard_normal(k).astype(np.float32)
    exact = oc.contract(A, "k", (k,), B, "k", (k,), "")
    mag = oc.magnitude(A, "k", (k,), B, "k", (k,), "")
    bound = oc.error_bound(mag, k, "f32")
    for order in (np.arange(k), np.argsort(np.abs(A * B))[::-1], rng.permutation(k)):
        s = np.float32(0)
        for i in order:
            s = np.float32(s + np.float32(A[i] * B[i]))
        assert abs(float(s) - exact[0]) <= bound[0]


_MUTANTS = {
    "c_order": ('order="F")', 'order="C")'),
    "beta_dropped": ("float(beta) * _tensor(C, size_c)", "0.0 * _tensor(C, size_c)"),
    "alpha_squared": ("out = float(alpha) * prod", "out = float(alpha) ** 2 * prod"),
    "modes_swapped": ('f"{modes_a},{modes_b}->{modes_c}"', 'f"{modes_b},{modes_a}->{modes_c[::-1]}"'),
}


@pytest.mark.parametrize("name", sorted(_MUTANTS))
def test_mutants_are_caught(name, tmp_path):
    import importlib.util
    import inspect
    src = inspect.getsource(oc)
    old, new = _MUTANTS[name]
    assert old in src
    path = tmp_path / f"mutant_{name}.py"
    path.write_text(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location(f"mutant_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    caught = False
    for ma, sa, mb, sb, mc in CASES:
        rng = np.random.default_rng(9)
        A, B = _rand(rng, int(np.prod(sa))), _rand(rng, int(np.prod(sb)))
        ext = oc.extents(ma, sa, mb, sb)
        C = _rand(rng, int(np.prod([ext[m] for m in mc])))
        want = _brute(A, ma, sa, B, mb, sb, mc, 1.5, 0.5, C)
        try:
            got = mod.contract(A, ma, sa, B, mb, sb, mc, 1.5, 0.5, C)
        except Exception:
            caught = True
            break
        if got.shape != want.shape or not np.array_equal(got, want):
            caught = True
            break
    assert caught, name
