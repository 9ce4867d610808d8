"""The autotune path's candidate plans (Section 3.1): every plan the tuner
may launch is built on the CPU and run through the host emulator -- on small
ragged problems against the oracle bit for bit, and at the full workload
sizes as a dry run of bounds, alignment and coverage -- before any of them
is timed on a GPU."""
from __future__ import annotations

import itertools

import numpy as np
import pytest

from oracle import oracle as orc
from paper_1704_04374_amd import hptt
from paper_1704_04374_amd.workloads import SUBTENSOR_WORKLOADS, WORKLOADS
from emulator import emu

ALL = WORKLOADS + SUBTENSOR_WORKLOADS

# Small problems of each kernel class, with ragged edges in every index.
SMALL = [
    ((97, 65, 33), (2, 0, 1), 1.0, 0.0, "f32"),
    ((1000, 1032), (1, 0), 1.5, 0.0, "f32"),
    ((300, 257), (1, 0), -0.5, 1.25, "f64"),
    ((7, 9, 6, 11, 5, 8), (5, 2, 0, 4, 1, 3), 1.5, 0.0, "f32"),
    ((3, 2, 40, 33, 17), (4, 2, 0, 3, 1), 1.0, 1.0, "f32"),
    ((24, 13, 9, 10), (0, 3, 2, 1), 2.0, 0.5, "f64"),
    ((63, 13, 9), (0, 2, 1), 1.0, 1.0, "f32"),
    ((4100,), (0,), 2.0, 0.5, "f32"),
]


def _rand(rng, n, dtype):
    return (rng.integers(-(1 << 20), 1 << 20, size=n) / float(1 << 20)).astype(dtype)


def _knobs(opt: dict) -> dict:
    return {k: v for k, v in opt.items() if v}


def test_quick_plan_comes_first_and_candidates_are_distinct():
    for w in ALL:
        cands = hptt.autotune_candidates(w.perm, w.size_a, w.alpha, w.beta, w.dtype,
                                         w.outer_a, w.outer_b)
        assert cands and not _knobs(cands[0]), w.name
        assert len(cands) <= 256
        plans = set()
        for c in cands:
            p = hptt.Plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype, outer_size_a=w.outer_a,
                          outer_size_b=w.outer_b, **_knobs(c))
            key = (p.describe(), p.info["hints"], p.info["tile_order"])
            assert key not in plans, (w.name, c)
            plans.add(key)
        kernel = hptt.Plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype,
                           outer_size_a=w.outer_a, outer_size_b=w.outer_b).info["kernel"]
        if kernel == "tile":
            assert len(cands) > 10, w.name


def test_candidates_reject_invalid_problems():
    with pytest.raises(hptt.HpttError):
        hptt.autotune_candidates((0, 0), (4, 4))
    with pytest.raises(hptt.HpttError):
        hptt.autotune_candidates((1, 0), (4, 4), outer_size_a=(3, 4))


def test_candidate_count_without_output_buffer():
    w = WORKLOADS[1]
    full = hptt.autotune_candidates(w.perm, w.size_a, w.alpha, w.beta, w.dtype)
    few = hptt.autotune_candidates(w.perm, w.size_a, w.alpha, w.beta, w.dtype, max_options=3)
    assert few == full[:3]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "x".join(map(str, c[0])))
def test_every_candidate_matches_oracle(case):
    size_a, perm, alpha, beta, dtype = case
    rng = np.random.default_rng(sum(size_a))
    npd = np.float32 if dtype == "f32" else np.float64
    n = int(np.prod(size_a))
    A = _rand(rng, n, npd)
    B0 = _rand(rng, n, npd) if beta != 0 else np.full(n, np.nan, npd)
    want = orc.transpose(A, size_a, perm, alpha, beta, B0 if beta != 0 else None)
    for c in hptt.autotune_candidates(perm, size_a, alpha, beta, dtype):
        p = emu.plan(perm, size_a, alpha, beta, dtype, **_knobs(c))
        B = B0.copy()
        err, msg, cnt = emu.run(p, A, B, counts=True)
        assert err == 0, f"{c}: {p.describe()}: {msg}"
        assert np.all(cnt == 1), f"{c}: {p.describe()}"
        assert np.array_equal(B, want), f"{c}: {p.describe()}"


def test_timing_plans_are_valid():
    """The tuner times each candidate with alpha = 0, beta = 1: that plan
    must be as valid as the user's, and leave B bit for bit unchanged."""
    size_a, perm = (97, 65, 33), (2, 0, 1)
    rng = np.random.default_rng(5)
    n = int(np.prod(size_a))
    A = _rand(rng, n, np.float32)
    B0 = _rand(rng, n, np.float32)
    B0[B0 == 0] = 0.25      # -0.0 would come back as +0.0
    for c in hptt.autotune_candidates(perm, size_a, 1.0, 0.0, "f32"):
        p = emu.plan(perm, size_a, 0.0, 1.0, "f32", **_knobs(c))
        B = B0.copy()
        err, msg, cnt = emu.run(p, A, B, counts=True)
        assert err == 0 and np.all(cnt == 1), f"{c}: {msg}"
        assert np.array_equal(B.view(np.uint32), B0.view(np.uint32)), c


@pytest.mark.parametrize("w", ALL, ids=lambda w: w.name)
def test_every_candidate_full_size_dry_run(w):
    """Every candidate at its workload's full size: a strided sample of the
    workgroups checks bounds and alignment (and that nothing is written
    twice); three seeded candidates are run whole, every B element written
    exactly once (inside the sub-tensor, never outside it)."""
    cands = hptt.autotune_candidates(w.perm, w.size_a, w.alpha, w.beta, w.dtype,
                                     w.outer_a, w.outer_b)
    rng = np.random.default_rng(len(cands))
    whole = set(int(i) for i in rng.choice(len(cands), size=min(3, len(cands)), replace=False))
    # the tuner times beta = 0 plans as they are (into a scratch tensor) and
    # others with alpha = 0, beta = 1 (also beta = 0 plans when it has no
    # memory for the scratch tensor)
    modes = ([(w.alpha, w.beta)] if w.beta == 0 else []) + [(0.0, 1.0)]
    for (i, c), (j, (alpha, beta)) in itertools.product(enumerate(cands), enumerate(modes)):
        p = emu.plan(w.perm, w.size_a, alpha, beta, w.dtype, outer_size_a=w.outer_a,
                     outer_size_b=w.outer_b, **_knobs(c))
        stride = 1 if (i in whole and j == 0) else max(1, p.info["grid"] // 97)
        err, msg, cnt = emu.run(p, counts=True, block_stride=stride)
        assert err == 0, f"{c}: {p.describe()}: {msg}"
        assert cnt.max() <= 1, f"{c}: {p.describe()}"
        if stride == 1:
            if w.outer_b is None:
                assert cnt.min() == 1, f"{c}: {p.describe()}"
            else:
                assert int(cnt.sum()) == w.numel, f"{c}: {p.describe()}"
