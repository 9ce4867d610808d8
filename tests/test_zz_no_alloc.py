"""The allocation-free contraction entry point (hptt_contraction_exec_no_alloc)
against the allocating one (hptt_contraction_exec) on an MI355X, through the
contraction C ABI: two calls in a row, the second on a smaller problem, each
compared with the allocating entry point's result on the same tensors and with
the contraction oracle.

Bar: the same as the contraction tests -- every element within
(k + 2) u (|alpha| sum |A||B| + |beta| |C|) of the exact value -- and the two
entry points within twice that of each other (they run the same kernels and
GEMM, so in practice they agree bit for bit, which is reported)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import contract as oc
from paper_1704_04374_amd import contraction, hptt
from paper_1704_04374_amd.contraction import Contraction

pytestmark = pytest.mark.gpu

NP = {"f32": np.float32, "f64": np.float64}


def _case(spec, ext, alpha, beta, dtype, seed):
    mc, ab = spec.split("=")
    ma, mb = ab.split("*")
    sa, sb = [ext[m] for m in ma], [ext[m] for m in mb]
    sc = [ext[m] for m in mc]
    rng = np.random.default_rng(seed)
    A = rng.uniform(-1, 1, int(np.prod(sa))).astype(NP[dtype])
    B = rng.uniform(-1, 1, int(np.prod(sb))).astype(NP[dtype])
    C0 = rng.uniform(-1, 1, int(np.prod(sc))).astype(NP[dtype])
    p = Contraction(mc, ma, sa, mb, sb, alpha, beta, dtype)
    return p, (ma, sa, A), (mb, sb, B), (mc, C0)


def _run_pair(p, a, b, c, dtype):
    (ma, sa, A), (mb, sb, B), (mc, C0) = a, b, c
    info = p.info
    print(f"[no_alloc] {p.describe()} workspace {info['workspace_bytes']}", flush=True)
    assert 0 < info["workspace_bytes"] <= contraction.STATIC_BYTES - contraction.STATIC_BLAS_BYTES
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    c_ref = torch.from_numpy(C0).cuda()
    c_new = torch.from_numpy(C0).cuda()
    p.exec(dA, dB, c_ref)
    p.exec_no_alloc(dA, dB, c_new)
    torch.cuda.synchronize()
    ref, new = c_ref.cpu().numpy(), c_new.cpu().numpy()
    exact = oc.contract(A, ma, sa, B, mb, sb, mc, p.alpha, p.beta, C0)
    mag = oc.magnitude(A, ma, sa, B, mb, sb, mc, p.alpha, p.beta, C0)
    bound = oc.error_bound(mag, info["gemm_k"], dtype)
    for name, got in (("exec", ref), ("exec_no_alloc", new)):
        err = np.abs(got.astype(np.float64) - exact)
        assert (err <= bound).all(), f"{name}: {int((err > bound).sum())} elements off"
    diff = np.abs(new.astype(np.float64) - ref.astype(np.float64))
    assert (diff <= 2 * bound).all()
    print(f"[no_alloc] bit-identical to exec: {np.array_equal(new, ref)}", flush=True)


def test_no_alloc_matches_exec_twice_second_smaller():
    # every operand and the product transposed (A, B and C all go through the array)
    p1, a1, b1, c1 = _case("acbd=aebf*dfce", dict(a=40, b=36, c=44, d=32, e=3, f=5),
                           0.75, 1.25, "f64", 1)
    assert all(p1.info[k] for k in ("transpose_a", "transpose_b", "transpose_c"))
    _run_pair(p1, a1, b1, c1, "f64")
    # a smaller problem next: the array keeps the first call's larger contents
    p2, a2, b2, c2 = _case("abc=bda*dc", dict(a=33, b=17, c=29, d=6), -1.5, 0.5, "f32", 2)
    assert p2.info["workspace_bytes"] < p1.info["workspace_bytes"]
    _run_pair(p2, a2, b2, c2, "f32")


def test_no_alloc_refuses_plans_beyond_the_array():
    # the transposed 56^4 fp64 product alone needs 75 MiB
    big = Contraction("acbd", "aebf", (56, 2, 56, 2), "dfce", (56, 2, 56, 2), 1.0, 0.0, "f64")
    assert big.info["workspace_bytes"] > contraction.STATIC_BYTES - contraction.STATIC_BLAS_BYTES
    A = torch.zeros(56 * 2 * 56 * 2, dtype=torch.float64, device="cuda")
    B = torch.zeros(56 * 2 * 56 * 2, dtype=torch.float64, device="cuda")
    C = torch.full((56 ** 4,), 3.0, dtype=torch.float64, device="cuda")
    with pytest.raises(hptt.HpttError) as e:
        big.exec_no_alloc(A, B, C)
    assert e.value.status == 2                    # HPTT_ERROR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((C == 3.0).all())                 # nothing was queued
