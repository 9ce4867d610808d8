"""Contractions by transposition - GEMM - transposition on an MI355X,
through the contraction C ABI, against the contraction oracle.

Bar: the GEMM sums the products in its own order, so results are not
bit-exact; every element must lie within (k + 2) u (|alpha| sum |A||B| +
|beta| |C|) of the exact value (u = 2^-24 for fp32, 2^-53 for fp64, k the
contraction length) -- the first-order bound of a dot product summed in any
order, plus the roundings of the alpha and beta products and the final sum."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import contract as oc
from paper_1704_04374_amd.contraction import Contraction
from paper_1704_04374_amd.workloads import CONTRACTIONS

pytestmark = pytest.mark.gpu

TORCH = {"f32": torch.float32, "f64": torch.float64}
NP = {"f32": np.float32, "f64": np.float64}


def _rand(rng, n, dtype):
    return rng.uniform(-1, 1, size=n).astype(NP[dtype])


def _check(got, exact, mag, k, dtype, what):
    bound = oc.error_bound(mag, k, dtype)
    err = np.abs(got.astype(np.float64) - exact)
    bad = np.flatnonzero(err > bound)
    assert bad.size == 0, (f"{what}: {bad.size} elements outside the bound, first at {bad[0]}: "
                           f"got {got[bad[0]]!r} exact {exact[bad[0]]!r} bound {bound[bad[0]]:.3e}")


def _random_spec(rng):
    """A random contraction over up to 7 modes with small extents."""
    letters = "abcdefg"
    n = int(rng.integers(2, 8))
    modes = list(letters[:n])
    roles = rng.integers(0, 4, size=n)       # 0: M, 1: N, 2: K, 3: batch
    a = [m for m, r in zip(modes, roles) if r in (0, 2, 3)]
    b = [m for m, r in zip(modes, roles) if r in (1, 2, 3)]
    c = [m for m, r in zip(modes, roles) if r in (0, 1, 3)]
    for x in (a, b, c):
        rng.shuffle(x)
    ext = {m: int(rng.choice([1, 2, 3, 5, 8, 13, 16])) for m in modes}
    return "".join(c), "".join(a), "".join(b), ext


def test_random_contractions():
    rng = np.random.default_rng(1704)
    cases = 0
    while cases < 120:
        mc, ma, mb, ext = _random_spec(rng)
        if not ma or not mb:
            continue
        dtype = ("f32", "f64")[cases % 2]
        alpha, beta = [(1.0, 0.0), (-1.5, 0.0), (0.75, 1.25), (1.0, -1.0)][cases % 4]
        sa, sb = [ext[m] for m in ma], [ext[m] for m in mb]
        p = Contraction(mc, ma, sa, mb, sb, alpha, beta, dtype)
        print(f"[contract] {p.describe()} alpha={alpha} beta={beta}", flush=True)
        A, B = _rand(rng, int(np.prod(sa)), dtype), _rand(rng, int(np.prod(sb)), dtype)
        nc = int(np.prod([ext[m] for m in mc]))
        C0 = _rand(rng, nc, dtype)
        exact = oc.contract(A, ma, sa, B, mb, sb, mc, alpha, beta, C0)
        mag = oc.magnitude(A, ma, sa, B, mb, sb, mc, alpha, beta, C0)
        dA, dB, dC = (torch.from_numpy(x).cuda() for x in (A, B, C0))
        p.exec(dA, dB, dC)
        torch.cuda.synchronize()
        _check(dC.cpu().numpy(), exact, mag, p.info["gemm_k"], dtype, p.describe())
        cases += 1


@pytest.mark.parametrize("w", CONTRACTIONS, ids=lambda w: w.name)
def test_contraction_workloads(w):
    """Each benchmark contraction at its full size (sampled elements), and
    again with beta != 0 so that every transposed C path adds beta * C."""
    print(f"[contract] {w.name}: {w.spec} {dict(w.extents)}", flush=True)
    rng = np.random.default_rng(w.seed + 7)
    sa, sb = w.size(w.modes_a), w.size(w.modes_b)
    A = _rand(rng, w.numel(w.modes_a), w.dtype)
    B = _rand(rng, w.numel(w.modes_b), w.dtype)
    C0 = _rand(rng, w.numel(w.modes_c), w.dtype)
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    offs = np.concatenate([[0, C0.size - 1], rng.integers(0, C0.size, 300)])
    for alpha, beta in ((w.alpha, w.beta), (-0.5, 2.0)):
        p = Contraction(w.modes_c, w.modes_a, sa, w.modes_b, sb, alpha, beta, w.dtype)
        dC = torch.from_numpy(C0).cuda()
        p.exec(dA, dB, dC)
        torch.cuda.synchronize()
        got = dC[torch.from_numpy(offs).cuda()].cpu().numpy()
        exact, mag = oc.contract_sample(A, w.modes_a, sa, B, w.modes_b, sb, w.modes_c, offs,
                                        alpha, beta, C0)
        _check(got, exact, mag, p.info["gemm_k"], w.dtype, p.describe())
        del dC


def test_workspace_and_stream():
    """A plan runs on a side stream with a caller-sized workspace; a short
    workspace is refused before anything is queued."""
    rng = np.random.default_rng(5)
    p = Contraction("abcd", "aebf", (8, 3, 8, 5), "dfce", (6, 5, 7, 3))
    need = p.info["workspace_bytes"]
    assert need > 0
    A, B = _rand(rng, 8 * 3 * 8 * 5, "f64"), _rand(rng, 6 * 5 * 7 * 3, "f64")
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    dC = torch.zeros(8 * 8 * 7 * 6, dtype=torch.float64, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        p.exec(dA, dB, dC, stream=s)
    s.synchronize()
    exact = oc.contract(A, "aebf", (8, 3, 8, 5), B, "dfce", (6, 5, 7, 3), "abcd")
    mag = oc.magnitude(A, "aebf", (8, 3, 8, 5), B, "dfce", (6, 5, 7, 3), "abcd")
    _check(dC.cpu().numpy(), exact, mag, 15, "f64", p.describe())
    import ctypes
    from paper_1704_04374_amd import contraction, hptt
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    st = contraction.library().hptt_contraction_exec(
        p._handle, ctypes.c_void_p(dA.data_ptr()), ctypes.c_void_p(dB.data_ptr()),
        ctypes.c_void_p(dC.data_ptr()), ctypes.c_void_p(ws.data_ptr()), need - 1,
        ctypes.c_void_p(0))
    assert st == 1   # HPTT_ERROR_INVALID_ARGUMENT
    assert hptt.SUCCESS == 0
