"""The contraction planner (transposition - GEMM - transposition) on the CPU:
which operands it transposes, the GEMM shape it forms, the workspace it
asks for, and the problems it rejects.  Plan creation makes no HIP call."""
from __future__ import annotations

import numpy as np
import pytest

from paper_1704_04374_amd import hptt
from paper_1704_04374_amd.contraction import Contraction


def _plan(spec, ext, **kw):
    c, rest = spec.split("=")
    a, b = rest.split("*")
    return Contraction(c, a, [ext[m] for m in a], b, [ext[m] for m in b], **kw)


EXT = dict(a=6, b=5, c=4, d=3, e=7, f=2, i=9, j=8, k=10, l=3)


@pytest.mark.parametrize("spec,ta,tb,tc,swap", [
    ("ij=ik*kj", 0, 0, 0, 0),        # plain matrix product
    ("ij=ki*kj", 0, 0, 0, 0),        # A read transposed in place
    ("ij=ik*jk", 0, 0, 0, 0),        # B read transposed in place
    ("ji=ik*kj", 0, 0, 0, 1),        # C = (A B)^T: formed as B^T A^T
    ("ijl=ikl*kjl", 0, 0, 0, 0),     # batched
    ("abcd=aebf*dfce", 1, 1, 0, 0),  # both inputs transposed, C in place
    ("abc=acd*db", 0, 0, 1, 0),      # C interleaves row and column modes
    ("cab=ak*kbc", 0, 0, 1, 0),      # C's modes interleave A's and B's
])
def test_transposes_only_what_gemm_cannot_read(spec, ta, tb, tc, swap):
    p = _plan(spec, EXT)
    i = p.info
    assert (i["transpose_a"], i["transpose_b"], i["transpose_c"]) == (ta, tb, tc), p.describe()
    if not tc:
        assert i["swap"] == swap, p.describe()


def test_gemm_shape_and_workspace():
    p = _plan("abcd=aebf*dfce", EXT, dtype="f64")
    i = p.info
    a, b, c, d, e, f = (EXT[m] for m in "abcdef")
    assert (i["gemm_m"], i["gemm_n"], i["gemm_k"], i["batch"]) == (a * b, c * d, e * f, 1)
    assert i["flops"] == 2.0 * a * b * c * d * e * f
    ab = lambda n: (n * 8 + 255) // 256 * 256
    assert i["workspace_bytes"] == ab(a * e * b * f) + ab(d * f * c * e)
    assert i["bytes_transposed"] == 8 * 2 * (a * e * b * f + d * f * c * e)
    q = _plan("ijl=ikl*kjl", EXT)
    assert q.info["workspace_bytes"] == 0 and q.info["batch"] == EXT["l"]


def test_scalar_and_outer_products():
    dot = _plan("=k*k", EXT)
    assert (dot.info["gemm_m"], dot.info["gemm_n"], dot.info["gemm_k"]) == (1, 1, EXT["k"])
    outer = _plan("ij=i*j", EXT)
    assert (outer.info["gemm_m"], outer.info["gemm_n"], outer.info["gemm_k"]) == (9, 8, 1)
    assert outer.info["workspace_bytes"] == 0


def test_cheapest_arrangement_is_chosen():
    """C is the largest tensor: transposing both (small) inputs beats
    transposing C."""
    ext = dict(a=64, b=64, c=64, d=64, e=4, f=4)
    p = _plan("abcd=aebf*dfce", ext)
    assert not p.info["transpose_c"]
    # when C is small and the inputs large, C is the one to transpose
    ext = dict(a=4, b=4, k=4096, c=3)
    q = _plan("bac=kab*kc", ext)
    assert not q.info["transpose_a"] and not q.info["transpose_b"], q.describe()


@pytest.mark.parametrize("bad", [
    ("ab", (2, 2), "bb", (2, 2), "a"),     # repeated mode
    ("ab", (2, 3), "bc", (4, 5), "ac"),    # extents disagree
    ("ab", (2, 3), "bc", (3, 5), "acz"),   # a mode of C from nowhere
    ("abx", (2, 3, 2), "bc", (3, 5), "ac"),  # a mode of A summed alone
    ("ab", (2, 0), "bc", (0, 5), "ac"),    # empty extent
])
def test_invalid_problems(bad):
    a, sa, b, sb, c = bad
    with pytest.raises(hptt.HpttError):
        Contraction(c, a, sa, b, sb)


def _gemm_colmajor(op_p, op_q, m, n, k, alpha, P, ldp, sp, Q, ldq, sq, beta, C, ldc, sc, batch):
    """A column-major strided-batched GEMM as BLAS defines it, reading and
    writing only through explicit offsets, each checked against its buffer."""
    for b in range(batch):
        ip = np.arange(m)[:, None] * (ldp if op_p else 1) + np.arange(k)[None, :] * (1 if op_p else ldp)
        iq = np.arange(k)[:, None] * (ldq if op_q else 1) + np.arange(n)[None, :] * (1 if op_q else ldq)
        ic = np.arange(m)[:, None] + np.arange(n)[None, :] * ldc
        for idx, buf in ((ip + b * sp, P), (iq + b * sq, Q), (ic + b * sc, C)):
            assert idx.min() >= 0 and idx.max() < buf.size, "GEMM access out of bounds"
        prod = P[ip + b * sp] @ Q[iq + b * sq]
        C[ic + b * sc] = alpha * prod + (beta * C[ic + b * sc] if beta else 0.0)


def _transpose(x, src, dst, ext):
    from oracle import oracle as orc
    if src == dst:
        return x.copy()
    return orc.transpose(x, [ext[m] for m in src], [src.index(m) for m in dst], 1.0, 0.0, None)


def _simulate(p, A, B, C0, ext):
    """Execute a plan's recipe on the CPU from its published shape: the
    transpositions it names (by the transposition oracle), the GEMM with its
    leading dimensions and strides (bounds-checked), the final transposition
    adding beta * C."""
    i = p.info
    x, y, k, l = i["modes_x"], i["modes_y"], i["modes_k"], i["modes_l"]
    swap = i["swap"]
    Pm, Qm = (p.modes_b, p.modes_a) if swap else (p.modes_a, p.modes_b)
    P, Q = (B, A) if swap else (A, B)
    if (i["transpose_b"] if swap else i["transpose_a"]):
        P = _transpose(P, Pm, x + k + l, ext)
    else:
        assert Pm == (k + x + l if i["op_p"] else x + k + l)
    if (i["transpose_a"] if swap else i["transpose_b"]):
        Q = _transpose(Q, Qm, k + y + l, ext)
    else:
        assert Qm == (y + k + l if i["op_q"] else k + y + l)
    if i["transpose_c"]:
        Cg = np.zeros(i["stride_c"] * i["batch"])
        _gemm_colmajor(i["op_p"], i["op_q"], i["gemm_m"], i["gemm_n"], i["gemm_k"], p.alpha, P,
                       i["ld_p"], i["stride_p"], Q, i["ld_q"], i["stride_q"], 0.0, Cg, i["ld_c"],
                       i["stride_c"], i["batch"])
        from oracle import oracle as orc
        src = x + y + l
        return orc.transpose(Cg, [ext[m] for m in src], [src.index(m) for m in p.modes_c], 1.0,
                             p.beta, C0 if p.beta else None)
    assert p.modes_c == x + y + l
    C = C0.copy()
    _gemm_colmajor(i["op_p"], i["op_q"], i["gemm_m"], i["gemm_n"], i["gemm_k"], p.alpha, P,
                   i["ld_p"], i["stride_p"], Q, i["ld_q"], i["stride_q"], p.beta, C, i["ld_c"],
                   i["stride_c"], i["batch"])
    return C


def test_plan_recipe_matches_oracle_on_cpu():
    """Random contractions of every role mix: the plan's transpositions, GEMM
    shape, leading dimensions and strides, replayed on the CPU, give the
    oracle's result and never index outside a buffer."""
    from oracle import contract as oc
    rng = np.random.default_rng(2017)
    letters = "abcdefg"
    done = 0
    while done < 300:
        n = int(rng.integers(1, 8))
        modes = list(letters[:n])
        roles = rng.integers(0, 4, size=n)
        a = [m for m, r in zip(modes, roles) if r in (0, 2, 3)]
        b = [m for m, r in zip(modes, roles) if r in (1, 2, 3)]
        c = [m for m, r in zip(modes, roles) if r in (0, 1, 3)]
        if not a or not b:
            continue
        for t in (a, b, c):
            rng.shuffle(t)
        a, b, c = "".join(a), "".join(b), "".join(c)
        ext = {m: int(rng.choice([1, 2, 3, 4, 5])) for m in modes}
        alpha, beta = [(1.0, 0.0), (0.5, -2.0)][done % 2]
        p = Contraction(c, a, [ext[m] for m in a], b, [ext[m] for m in b], alpha, beta)
        A = rng.integers(-4, 4, size=int(np.prod([ext[m] for m in a]))).astype(np.float64)
        B = rng.integers(-4, 4, size=int(np.prod([ext[m] for m in b]))).astype(np.float64)
        C0 = rng.integers(-4, 4, size=int(np.prod([ext[m] for m in c]))).astype(np.float64)
        got = _simulate(p, A, B, C0, ext)
        want = oc.contract(A, a, [ext[m] for m in a], B, b, [ext[m] for m in b], c, alpha, beta, C0)
        assert np.array_equal(got, want), p.describe()
        done += 1


def _steps(p, ext):
    """(source modes, target modes, alpha, beta) of each transposition a plan runs."""
    i = p.info
    x, y, k, l = i["modes_x"], i["modes_y"], i["modes_k"], i["modes_l"]
    Pm, Qm = (p.modes_b, p.modes_a) if i["swap"] else (p.modes_a, p.modes_b)
    out = []
    if i["transpose_b"] if i["swap"] else i["transpose_a"]:
        out.append((Pm, x + k + l, 1.0, 0.0))
    if i["transpose_a"] if i["swap"] else i["transpose_b"]:
        out.append((Qm, k + y + l, 1.0, 0.0))
    if i["transpose_c"]:
        out.append((x + y + l, p.modes_c, 1.0, p.beta))
    return out


def test_workload_transpositions_dry_run():
    """Every transposition the benchmark contractions launch, at full size,
    through the host emulator (strided sample of workgroups)."""
    from emulator import emu
    from paper_1704_04374_amd.workloads import CONTRACTIONS
    for w in CONTRACTIONS:
        ext = w.ext()
        for beta in (w.beta, 2.0):
            p = Contraction(w.modes_c, w.modes_a, w.size(w.modes_a), w.modes_b,
                            w.size(w.modes_b), w.alpha, beta, w.dtype)
            for src, dst, al, be in _steps(p, ext):
                t = emu.plan([src.index(m) for m in dst], [ext[m] for m in src], al, be, w.dtype)
                err, msg, _ = emu.run(t, block_stride=max(1, t.info["grid"] // 101))
                assert err == 0, (w.name, src, dst, msg)
