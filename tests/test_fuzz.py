"""Randomised parity: seeded random problems (tests/fuzz_cases.py) through
the bounds-checking host emulator on the CPU, and the same problems on the
GPU against the oracle, bit-exact, over the whole buffers (the elements
outside a sub-tensor, and before the pointers, must come back unchanged)."""
from __future__ import annotations

import numpy as np
import pytest

import fuzz_cases as fc
from paper_1704_04374_amd import hptt

SETS = [(7, 1500), (8, 1500)]  # (seed, cases): set 7 allows extent-1 indices freely


def _cases():
    for seed, n in SETS:
        for i in range(n):
            yield seed, i, fc.case(seed, i)


def _plan(lib_plan, c):
    return lib_plan(c["perm"], c["size"], c["alpha"], c["beta"], c["dtype"], **fc.plan_kwargs(c))


def _aligned_width(v, off):
    while v > 1 and off % v:
        v //= 2
    return v


def test_fuzz_cases_in_bounds():
    """Every access in bounds and aligned as its width requires, every B
    element of a compact B written once, in the variant and widths hptt_exec
    would launch for the pointers' offsets."""
    from emulator import emu
    ran = 0
    for seed, i, c in _cases():
        try:
            p = _plan(emu.plan, c)
        except hptt.HpttError:
            continue  # an option combination the plan builder rejects
        info = p.info
        if info["kernel"] == "none":
            continue
        a0, b0, _, _ = fc.first_elements(c)
        if info["kernel"] == "tile":
            kw = dict(mis_a=a0 % info["vec_a"], mis_b=b0 % info["vec_b"])
        else:
            kw = dict(va=_aligned_width(info["vec_a"], a0), vb=_aligned_width(info["vec_b"], b0))
        err, msg, cnt = emu.run(p, counts=not c["outer"], **kw)
        assert err == 0, f"set {seed} case {i} {c}: {msg} ({p.describe()})"
        if cnt is not None:
            assert cnt.min() == 1 and cnt.max() == 1, f"set {seed} case {i} {c}: {p.describe()}"
        ran += 1
    assert ran >= 2500


@pytest.mark.gpu
def test_fuzz_cases_match_oracle():
    import torch
    from oracle import oracle as orc
    npd = {"f32": np.float32, "f64": np.float64}
    ran = 0
    for seed, i, c in _cases():
        try:
            p = _plan(hptt.create_plan, c)
        except hptt.HpttError:
            continue
        if p.info["kernel"] == "none":
            continue
        rng = np.random.default_rng([seed, i, 1])
        a0, b0, na, nb = fc.first_elements(c)
        A = (rng.integers(-(1 << 20), 1 << 20, size=na) / float(1 << 20)).astype(npd[c["dtype"]])
        B = (rng.integers(-(1 << 20), 1 << 20, size=nb) / float(1 << 20)).astype(npd[c["dtype"]])
        if c["outer"]:
            tail = orc.transpose_outer(A[a0:], c["size"], c["perm"], c["outer"][0], c["outer"][1],
                                       c["alpha"], c["beta"], B[b0:])
        else:
            tail = orc.transpose(A[a0:], c["size"], c["perm"], c["alpha"], c["beta"],
                                 B[b0:] if c["beta"] != 0 else None)
        want = B.copy()
        want[b0:b0 + tail.size] = tail
        dA = torch.from_numpy(A).cuda()
        dB = torch.from_numpy(B).cuda()
        p.exec(dA[a0:], dB[b0:])
        torch.cuda.synchronize()
        got = dB.cpu().numpy()
        if not np.array_equal(got, want):
            bad = np.flatnonzero(got != want)
            raise AssertionError(f"set {seed} case {i} {c}: {bad.size} elements differ, first at "
                                 f"{bad[0]} ({p.describe()})")
        ran += 1
    assert ran >= 2500
