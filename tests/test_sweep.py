"""The seeded 57-case sweep that stands in for the paper's benchmark of 57
transpositions of 2-D to 6-D tensors of about 200 MB (Section 4): its shape,
and a host-emulator dry run of every plan it launches (the quick path's and
every autotune candidate), before any of them runs on a GPU."""
from __future__ import annotations

from collections import Counter
from math import prod

import numpy as np
import pytest

from paper_1704_04374_amd import hptt
from paper_1704_04374_amd.workloads import SWEEP_BYTES, SWEEP_DIMS, sweep57
from emulator import emu

CASES = sweep57()


def test_sweep_shape():
    assert len(CASES) == 57 and sum(SWEEP_DIMS.values()) == 57
    assert Counter(len(w.size_a) for w in CASES) == Counter(SWEEP_DIMS)
    assert len({w.name for w in CASES}) == 57
    for w in CASES:
        assert w.dtype == "f32" and w.beta != 0 and min(w.size_a) >= 2
        assert abs(w.tensor_bytes / SWEEP_BYTES - 1) <= 0.03
        assert sorted(w.perm) == list(range(len(w.perm))) and w.perm != tuple(range(len(w.perm)))
    assert [w.name for w in sweep57()] == [w.name for w in CASES]      # seeded
    assert [w.name for w in sweep57(seed=7)] != [w.name for w in CASES]


def _dry(p, stride):
    err, msg, cnt = emu.run(p, counts=stride == 1, block_stride=stride)
    assert err == 0, f"{p.describe()}: {msg}"
    if stride == 1:
        assert cnt.min() == 1 and cnt.max() == 1, p.describe()


@pytest.mark.parametrize("dims", sorted(SWEEP_DIMS))
def test_sweep_plans_dry_run(dims):
    """Every plan the sweep may launch: the quick plans for beta = 1 and
    beta = 0 and the timing plan of every autotune candidate, on a strided
    sample of workgroups; the quick plan of one case per dimension whole,
    every B element written exactly once."""
    ws = [w for w in CASES if len(w.size_a) == dims]
    whole = ws[dims % len(ws)]
    for w in ws:
        for alpha, beta in ((w.alpha, w.beta), (w.alpha, 0.0)):
            p = emu.plan(w.perm, w.size_a, alpha, beta, w.dtype)
            _dry(p, 1 if (w is whole and beta != 0) else max(1, p.info["grid"] // 89))
        for c in hptt.autotune_candidates(w.perm, w.size_a, w.alpha, w.beta, w.dtype):
            knobs = {k: v for k, v in c.items() if v}
            p = emu.plan(w.perm, w.size_a, 0.0, 1.0, w.dtype, **knobs)
            _dry(p, max(1, p.info["grid"] // 31))


def test_sweep_covers_kernel_classes():
    """The sweep reaches both kernel classes and the shared-run tiles."""
    seen, shared = set(), 0
    for w in CASES:
        p = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype)
        seen.add(p.info["kernel"])
        shared += p.info["shared_runs"] > 0
    assert {"tile", "stream"} <= seen
    assert shared >= 10
