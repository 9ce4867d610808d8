"""The kernels' index arithmetic, run on the CPU by the host emulator and
compared with the oracle (bit for bit), with every global and LDS access
bounds-checked and every B element counted.  Catches out-of-bounds and
coverage bugs before any kernel runs on a GPU."""
from __future__ import annotations

import itertools

import numpy as np
import pytest

from oracle import oracle as orc
from paper_1704_04374_amd import hptt
from paper_1704_04374_amd.workloads import WORKLOADS, random_problem
from emulator import emu

CASES = [(1.0, 0.0), (1.5, 0.0), (-0.3, 1.25), (2.0, 0.5), (0.0, 1.0)]


def _rand(rng, n, dtype):
    return (rng.integers(-(1 << 20), 1 << 20, size=n) / float(1 << 20)).astype(dtype)


def _check(p, size_a, perm, alpha, beta, dtype, rng, **run_kw):
    npd = np.float32 if dtype == "f32" else np.float64
    A = _rand(rng, p.numel, npd)
    B0 = _rand(rng, p.numel, npd) if beta != 0 else np.full(p.numel, np.nan, npd)
    want = orc.transpose(A, size_a, perm, alpha, beta, B0 if beta != 0 else None)
    B = B0.copy()
    err, msg, cnt = emu.run(p, A, B, counts=True, **run_kw)
    assert err == 0, f"{p.describe()}: {msg}"
    assert np.all(cnt == 1), f"{p.describe()}: B elements written {np.unique(cnt)} times"
    assert np.array_equal(B, want), p.describe()


@pytest.mark.parametrize("d", [1, 2, 3, 5, 7, 24, 96, 97, 640, 1000, 65536, 65537, 3840,
                               (1 << 31) - 1, 1 << 31, (1 << 31) + 1, (1 << 32) - 1])
def test_fast_division(d):
    lib = emu.library()
    top = 1 << 32
    for lo, hi in [(0, 1 << 16), (top - (1 << 16), top), (d * 977 % top, d * 977 % top + 4096)]:
        hi = min(hi, top)
        assert lib.hptt_emulate_check_fastdiv(d, lo, hi) == -1, (d, lo)


def test_fast_division_random_divisors():
    lib = emu.library()
    rng = np.random.default_rng(7)
    for d in rng.integers(1, 1 << 32, size=200):
        start = int(rng.integers(0, (1 << 32) - 2048))
        assert lib.hptt_emulate_check_fastdiv(int(d), start, start + 2048) == -1, d
        assert lib.hptt_emulate_check_fastdiv(int(d), (1 << 32) - 512, 1 << 32) == -1, d


def test_random_problems_match_oracle():
    """Seeded sweep of small odd shapes over every kernel class, with tails."""
    rng = np.random.default_rng(2017)
    for it in range(120):
        size_a, perm = random_problem(rng, max_dims=6, max_numel=40000)
        dtype = "f32" if it % 2 == 0 else "f64"
        alpha, beta = CASES[it % len(CASES)]
        p = emu.plan(perm, size_a, alpha, beta, dtype)
        _check(p, size_a, perm, alpha, beta, dtype, rng)


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_sheared_b_runs_match_oracle(dtype):
    """B runs sheared onto 128-byte lines (each column's run starts on the line
    at or below its chunk, lineB - 1 more rows staged): every element written
    once, bit-exact, for base pointers off the line by 0..3 elements."""
    rng = np.random.default_rng(31)
    seen = 0
    for size_a, perm in [((397, 125), (1, 0)), ((153, 10, 325), (2, 0, 1)), ((64, 300), (1, 0)),
                         ((33, 7, 261), (2, 1, 0)), ((130, 129), (1, 0)),
                         ((65, 33, 129), (2, 0, 1)), ((17, 3, 200), (2, 1, 0))]:
        for alpha, beta in ((1.0, 0.0), (1.5, -0.5)):
            p = emu.plan(perm, size_a, alpha, beta, dtype, shear=1)
            if p.info["shear"] == 0:
                continue
            seen += 1
            for mis in (0, 1, 3):
                _check(p, size_a, perm, alpha, beta, dtype, rng, mis_b=mis)
    assert seen >= 8


def test_sheared_full_size_geometry():
    """Dry runs of sweep cases whose B rows are not whole lines: sheared by
    default, every offset in bounds, every B element written once."""
    from paper_1704_04374_amd.workloads import sweep57
    n = 0
    for w in sweep57(beta=0.0):
        p = emu.plan(w.perm, w.size_a, 1.0, 0.0, "f32")
        if not p.info["shear"]:
            continue
        n += 1
        err, msg, cnt = emu.run(p, counts=True)
        assert err == 0, (w.name, msg)
        assert cnt.min() == 1 and cnt.max() == 1, w.name
        if n == 4:
            break
    assert n == 4


def test_general_tile_variant_on_every_plan():
    """The tile kernel's general and shifted variants are also correct on
    plans where hptt_exec launches another one."""
    rng = np.random.default_rng(2018)
    seen = 0
    for it in range(80):
        size_a, perm = random_problem(rng, max_dims=6, max_numel=40000)
        dtype = "f32" if it % 2 == 0 else "f64"
        alpha, beta = CASES[it % len(CASES)]
        p = emu.plan(perm, size_a, alpha, beta, dtype)
        if p.info["kernel"] != "tile":
            continue
        seen += 1
        _check(p, size_a, perm, alpha, beta, dtype, rng, variant="general")
        _check(p, size_a, perm, alpha, beta, dtype, rng, variant="shifted")
    assert seen >= 20


@pytest.mark.parametrize("knobs", [
    dict(kernel="generic"),
    dict(run_a=4, run_b=4),
    dict(run_a=3, run_b=5),
    dict(run_a=1, run_b=1),
    dict(max_blocks=3),
    dict(lds_pad=-1),
    dict(lds_pad=4),
    dict(max_vec=1),
    dict(max_vec=2),
    dict(store_hint=1),
    dict(load_hint=1, store_hint=1),
    dict(tile_order=1),
    dict(tile_order=3),
    dict(tile_order=4),
    dict(row_passes=2),
    dict(row_passes=3, max_blocks=7),
    dict(row_passes=5, run_a=8, run_b=40),
    dict(row_passes=1),
    dict(tile_order=3, max_blocks=16),
    dict(tile_order=3, max_blocks=5),
    dict(run_a=64, run_b=64),
    dict(run_a=512, run_b=8),
    dict(exact_runs=1, run_a=6, run_b=10),
    dict(block=1024),
    dict(block=1024, run_a=96, run_b=160),
    dict(block=1024, row_passes=2, max_blocks=9),
    dict(block=1024, tile_order=3),
    dict(skew=3),
    dict(skew=7, tile_order=3),
    dict(grid_order=1),
    dict(grid_order=2),
    dict(grid_order=3),
    dict(grid_order=3, tile_order=3, max_blocks=11),
])
def test_knobs_match_oracle(knobs):
    rng = np.random.default_rng(11)
    for it in range(40):
        size_a, perm = random_problem(rng, max_dims=5, max_numel=20000)
        dtype = "f32" if it % 3 else "f64"
        alpha, beta = CASES[it % len(CASES)]
        p = emu.plan(perm, size_a, alpha, beta, dtype, **knobs)
        _check(p, size_a, perm, alpha, beta, dtype, rng)


@pytest.mark.parametrize("va,vb", [(1, 1), (1, 4), (4, 1), (2, 2), (2, 4)])
@pytest.mark.parametrize("order", [1, 2])
def test_narrow_vectors_as_for_misaligned_pointers(va, vb, order):
    """hptt_exec narrows the vector widths for less aligned pointers."""
    rng = np.random.default_rng(13)
    for size_a, perm in [((64, 33), (1, 0)), ((24, 20, 16, 5), (3, 2, 0, 1)),
                         ((3, 2, 64, 7, 32), (4, 2, 0, 3, 1)), ((96, 7, 9), (0, 2, 1))]:
        p = emu.plan(perm, size_a, 1.5, 0.5, "f32", tile_order=order)
        _check(p, size_a, perm, 1.5, 0.5, "f32", rng, va=min(va, p.info["vec_a"]),
               vb=min(vb, p.info["vec_b"]))


def test_edge_tiles_and_tails():
    rng = np.random.default_rng(17)
    for size_a, perm in [((65, 65), (1, 0)), ((33, 17, 5), (2, 0, 1)), ((7, 130, 3), (1, 2, 0)),
                         ((5, 3, 65, 9), (3, 2, 0, 1)), ((129, 3), (1, 0)), ((17, 1, 33), (2, 1, 0))]:
        for dtype in ("f32", "f64"):
            p = emu.plan(perm, size_a, 1.0, 0.0, dtype)
            _check(p, size_a, perm, 1.0, 0.0, dtype, rng)


@pytest.mark.parametrize("w", WORKLOADS[:1], ids=lambda w: w.name)
def test_small_workload_matches_oracle(w):
    rng = np.random.default_rng(w.seed_a)
    p = emu.plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype)
    _check(p, w.size_a, w.perm, w.alpha, w.beta, w.dtype, rng)


@pytest.mark.parametrize("knobs", [dict(), dict(tile_order=1), dict(tile_order=3),
                                   dict(tile_order=4), dict(block=1024), dict(row_passes=3),
                                   dict(grid_order=1), dict(grid_order=3)],
                         ids=["default", "digit_order", "xcd_order", "xcd_digit_order",
                              "block1024", "three_passes", "outer_a_order", "outer_b_order"])
@pytest.mark.parametrize("w", WORKLOADS, ids=lambda w: w.name)
def test_full_size_geometry(w, knobs):
    """Dry run of every workgroup of each full-size workload: every offset in
    bounds and aligned, every B element written exactly once."""
    p = emu.plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype, **knobs)
    err, msg, cnt = emu.run(p, counts=True)
    assert err == 0, msg
    assert cnt.min() == 1 and cnt.max() == 1


def _fortran_offset(index, outer):
    off, stride = 0, 1
    for i, o in zip(index, outer):
        off += int(i) * stride
        stride *= int(o)
    return off


@pytest.mark.parametrize("knobs", [dict(), dict(kernel="generic"), dict(run_a=4, run_b=4),
                                   dict(max_vec=1), dict(tile_order=1)],
                         ids=["default", "generic", "small_tiles", "scalar", "digit_order"])
def test_outer_sizes_match_oracle(knobs):
    """Sub-tensors at random positions of larger tensors (Fig. 3's
    transpose-and-compact and transpose-and-scatter): bit-exact against the
    oracle, B elements outside the sub-tensor never written."""
    rng = np.random.default_rng(31)
    for it in range(60):
        n = int(rng.integers(1, 6))
        size_a = tuple(int(x) for x in rng.choice([1, 2, 3, 5, 8, 17, 33, 64], size=n))
        if np.prod(size_a) > 30000:
            continue
        perm = tuple(int(p) for p in rng.permutation(n))
        size_b = tuple(size_a[p] for p in perm)
        outer_a = tuple(s + int(rng.choice([0, 0, 1, 3, 8])) for s in size_a)
        outer_b = tuple(s + int(rng.choice([0, 0, 1, 3, 8])) for s in size_b)
        start_a = tuple(int(rng.integers(0, o - s + 1)) for s, o in zip(size_a, outer_a))
        start_b = tuple(int(rng.integers(0, o - s + 1)) for s, o in zip(size_b, outer_b))
        dtype = ("f32", "f64")[it % 2]
        alpha, beta = CASES[it % len(CASES)]
        try:
            p = emu.plan(perm, size_a, alpha, beta, dtype, outer_size_a=outer_a,
                         outer_size_b=outer_b, **knobs)
        except Exception:
            if "kernel" in knobs:
                continue
            raise
        npd = np.float32 if dtype == "f32" else np.float64
        oa, ob = _fortran_offset(start_a, outer_a), _fortran_offset(start_b, outer_b)
        fa, fb = p.info["footprint_a"], p.info["footprint_b"]
        PA = _rand(rng, int(np.prod(outer_a)), npd)
        PB = _rand(rng, int(np.prod(outer_b)), npd)
        want = orc.transpose_outer(PA[oa:], size_a, perm, outer_a, outer_b, alpha, beta, PB[ob:])
        A = np.ascontiguousarray(PA[oa:oa + fa])
        B = np.ascontiguousarray(PB[ob:ob + fb])
        err, msg, cnt = emu.run(p, A, B, counts=True)
        assert err == 0, f"{p.describe()}: {msg}"
        assert np.array_equal(B, want[:fb]), p.describe()
        # each sub-tensor element written once, nothing else written
        mask = np.zeros(fb, dtype=bool)
        idx = np.indices(size_b).reshape(n, -1)
        strides = np.cumprod((1,) + outer_b[:-1])
        mask[(idx * np.array(strides)[:, None]).sum(axis=0)] = True
        assert np.all(cnt[mask] == 1) and np.all(cnt[~mask] == 0), p.describe()


@pytest.mark.parametrize("mis", [(1, 0), (0, 3), (2, 1), (3, 2)], ids=lambda m: f"misA{m[0]}_misB{m[1]}")
def test_tile_runs_shifted_onto_the_vector_grid(mis):
    """Base pointers off the 16-byte grid: the tile kernel keeps its vector
    widths and shifts every run onto the grid, with partial vectors at both
    ends.  Bit-exact against the oracle; every vector access aligned."""
    rng = np.random.default_rng(100 + 4 * mis[0] + mis[1])
    seen = 0
    for it in range(80):
        size_a, perm = random_problem(rng, max_dims=5, max_numel=30000)
        dtype = "f32" if it % 2 == 0 else "f64"
        alpha, beta = CASES[it % len(CASES)]
        p = emu.plan(perm, size_a, alpha, beta, dtype)
        if p.info["kernel"] != "tile":
            continue
        seen += 1
        per = 4 if dtype == "f32" else 2
        _check(p, size_a, perm, alpha, beta, dtype, rng, mis_a=mis[0] % per, mis_b=mis[1] % per)
    assert seen >= 20


@pytest.mark.parametrize("knobs", [dict(depth=2), dict(depth=3), dict(depth=7),
                                   dict(depth=5, max_vec=2), dict(min_tile=64),
                                   dict(min_tile=1 << 16), dict(run_a=4, run_b=4, depth=9)],
                         ids=lambda k: "_".join(f"{a}{b}" for a, b in k.items()))
def test_stacked_tiles_match_oracle(knobs):
    """Tiles stacked along one more index (depth), forced or chosen by the
    minimum tile size, with ragged last stacks: bit-exact, each B element
    written once."""
    rng = np.random.default_rng(7 + sum(knobs.values()))
    stacked = 0
    for it in range(80):
        size_a, perm = random_problem(rng, max_dims=6, extents=(1, 2, 3, 5, 7, 9, 17, 33),
                                      max_numel=40000)
        dtype = "f32" if it % 2 == 0 else "f64"
        alpha, beta = CASES[it % len(CASES)]
        try:
            p = emu.plan(perm, size_a, alpha, beta, dtype, kernel="tile", **knobs)
        except hptt.HpttError:
            continue
        stacked += p.info["depth"] > 1
        _check(p, size_a, perm, alpha, beta, dtype, rng, mis_a=it % 3 % (4 if dtype == "f32" else 2))
    assert stacked >= 5 or "depth" not in knobs


def test_small_tiles_grow_or_stack():
    """Leading extents too short for the target runs: the planner lengthens
    the other run or stacks tiles until a workgroup round holds at least
    min_tile elements (when the grid stays large)."""
    for size, perm in [((4, 11, 385, 2952), (1, 0, 2, 3)), ((2, 26250, 4, 238), (1, 3, 0, 2)),
                       ((2, 3, 2, 995, 4188), (2, 3, 0, 1, 4)), ((184, 2, 135870), (1, 0, 2)),
                       ((70, 5, 98, 1458), (1, 0, 2, 3))]:
        p = hptt.Plan(perm, size, 1.0, 1.0, "f32")
        i = p.info
        assert i["run_a"] * i["run_b"] * i["depth"] >= 2048, p.describe()
        err, msg, _ = emu.run(emu.plan(perm, size, 1.0, 1.0, "f32"), block_stride=97)
        assert err == 0, msg


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_shared_run_tiles_match_oracle(dtype):
    """Tiles whose A run and B run share indices (kept short stride-1 index,
    small B stride-1 extents), forced wherever they apply, over every update
    mode and with base pointers off the vector grid (runs shifted onto it):
    bit-exact, each B element written once."""
    rng = np.random.default_rng(1704 + len(dtype))
    seen = chunked = 0
    for it in range(200):
        size_a, perm = random_problem(rng, max_dims=6, extents=(1, 2, 3, 4, 5, 7, 12, 17, 33, 40),
                                      max_numel=30000)
        alpha, beta = CASES[it % len(CASES)]
        try:
            p = emu.plan(perm, size_a, alpha, beta, dtype, shared_runs=1)
        except hptt.HpttError:
            continue
        if p.info["kernel"] != "tile" or p.info["shared_runs"] == 0:
            continue
        seen += 1
        chunked += p.info["tiles"] > 1
        per = 4 if dtype == "f32" else 2
        _check(p, size_a, perm, alpha, beta, dtype, rng, mis_a=it % per, mis_b=(it // 2) % per)
    assert seen >= 40 and chunked >= 20, (seen, chunked)


@pytest.mark.parametrize("knobs", [dict(run_a=8, run_b=8), dict(run_a=64, run_b=16),
                                   dict(run_a=3, run_b=200), dict(tile_order=1),
                                   dict(tile_order=3), dict(tile_order=4), dict(lds_pad=-1),
                                   dict(lds_pad=4), dict(max_vec=1), dict(max_blocks=7)],
                         ids=lambda k: "_".join(f"{a}{b}" for a, b in k.items()))
def test_shared_run_knobs_match_oracle(knobs):
    """Shared-run tiles under the run targets, tile orders, LDS padding,
    scalar vectors and a capped grid (workgroups looping over tiles)."""
    rng = np.random.default_rng(99 + len(knobs))
    seen = 0
    shapes = [((12, 3, 2, 23, 13), (2, 1, 4, 3, 0)), ((184, 2, 35), (1, 0, 2)),
              ((29, 12, 2, 7), (2, 0, 3, 1)), ((2, 601, 41), (0, 2, 1)),
              ((4, 2, 17, 3, 12), (2, 1, 3, 0, 4)), ((3267, 15), (1, 0)),
              ((2, 56, 30, 14), (2, 0, 3, 1)), ((4, 2, 82, 5, 7, 3), (0, 4, 2, 1, 5, 3)),
              ((14, 3582), (1, 0)), ((2, 26, 4, 23), (1, 3, 0, 2))]
    for it, (size_a, perm) in enumerate(shapes):
        dtype = ("f32", "f64")[it % 2]
        alpha, beta = CASES[it % len(CASES)]
        p = emu.plan(perm, size_a, alpha, beta, dtype, shared_runs=1, **knobs)
        if p.info["shared_runs"] == 0:
            continue
        seen += 1
        _check(p, size_a, perm, alpha, beta, dtype, rng)
    assert seen >= 5


def test_shared_run_outer_sizes_match_oracle():
    """Shared-run tiles on sub-tensors (outer sizes break the contiguity the
    runs rely on at random places)."""
    rng = np.random.default_rng(77)
    seen = 0
    for it in range(80):
        n = int(rng.integers(2, 6))
        size_a = tuple(int(x) for x in rng.choice([2, 3, 5, 8, 17, 33], size=n))
        if np.prod(size_a) > 30000:
            continue
        perm = tuple(int(p) for p in rng.permutation(n))
        size_b = tuple(size_a[p] for p in perm)
        outer_a = tuple(s + int(rng.choice([0, 0, 0, 1, 3])) for s in size_a)
        outer_b = tuple(s + int(rng.choice([0, 0, 0, 1, 3])) for s in size_b)
        dtype = ("f32", "f64")[it % 2]
        alpha, beta = CASES[it % len(CASES)]
        try:
            p = emu.plan(perm, size_a, alpha, beta, dtype, outer_size_a=outer_a,
                         outer_size_b=outer_b, shared_runs=1)
        except hptt.HpttError:
            continue
        if p.info["kernel"] != "tile" or p.info["shared_runs"] == 0:
            continue
        seen += 1
        npd = np.float32 if dtype == "f32" else np.float64
        fa, fb = p.info["footprint_a"], p.info["footprint_b"]
        PA = _rand(rng, int(np.prod(outer_a)), npd)
        PB = _rand(rng, int(np.prod(outer_b)), npd)
        want = orc.transpose_outer(PA, size_a, perm, outer_a, outer_b, alpha, beta, PB)
        A = np.ascontiguousarray(PA[:fa])
        B = np.ascontiguousarray(PB[:fb])
        err, msg, cnt = emu.run(p, A, B, counts=True)
        assert err == 0, f"{p.describe()}: {msg}"
        assert np.array_equal(B, want[:fb]), p.describe()
        mask = np.zeros(fb, dtype=bool)
        idx = np.indices(size_b).reshape(n, -1)
        strides = np.cumprod((1,) + outer_b[:-1])
        mask[(idx * np.array(strides)[:, None]).sum(axis=0)] = True
        assert np.all(cnt[mask] == 1) and np.all(cnt[~mask] == 0), p.describe()
    assert seen >= 15, seen


def test_shared_run_full_size_geometry():
    """Dry runs of sweep cases planned with shared runs by default (shared
    chunked index, chunked A-only and B-only indices, kept stride-1 index):
    every offset in bounds and aligned, every B element written once."""
    from paper_1704_04374_amd.workloads import sweep57
    names = ("sweep3d_05", "sweep3d_08", "sweep5d_00", "sweep5d_08", "sweep6d_11")
    n = 0
    for w in sweep57():
        if not w.name.startswith(names):
            continue
        p = emu.plan(w.perm, w.size_a, w.alpha, w.beta, "f32")
        assert p.info["kernel"] == "tile" and p.info["shared_runs"] >= 1, p.describe()
        n += 1
        err, msg, cnt = emu.run(p, counts=True)
        assert err == 0, (w.name, msg)
        assert cnt.min() == 1 and cnt.max() == 1, w.name
    assert n == len(names)


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_flat_b_runs_match_oracle(dtype):
    """Flat B runs (whole lines cut from the flattened range of two or more B
    indices, the row table rebuilt per tile): every element written once and
    bit-exact, in each tile variant, with misaligned base pointers and a
    partial last chunk."""
    rng = np.random.default_rng(1704)
    shapes = [((24, 6, 16, 20), (3, 2, 0, 1)), ((13, 5, 7, 9), (3, 2, 0, 1)),
              ((10, 3, 5, 7), (3, 2, 1, 0)), ((8, 4, 3, 20, 16), (4, 3, 0, 2, 1)),
              ((33, 2, 9, 11), (2, 3, 0, 1)), ((5, 40, 3, 6, 7), (4, 3, 2, 0, 1))]
    seen = 0
    for size_a, perm in shapes:
        for (alpha, beta), knobs in itertools.product(
                ((1.0, 0.0), (1.5, 0.0), (-0.3, 1.25)),
                (dict(), dict(run_b=8), dict(run_a=16, run_b=8))):
            p = emu.plan(perm, size_a, alpha, beta, dtype, flat_runs=1, **knobs)
            if not p.info["flat_runs"]:
                continue
            seen += 1
            for variant in (None, "shifted", "general"):
                for mis in ((0, 0), (1, 3)):
                    if variant is None and mis != (0, 0):
                        continue
                    _check(p, size_a, perm, alpha, beta, dtype, rng, variant=variant,
                           mis_a=mis[0], mis_b=mis[1])
    assert seen >= 9


def test_flat_b_runs_full_size_geometry():
    """The 6-D fp32 workload takes flat B runs by default; dry run of every
    workgroup at full size: in bounds, every B element written once."""
    w = [w for w in WORKLOADS if w.size_a == (24, 20, 16, 24, 18, 20)][0]
    p = emu.plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype)
    assert p.info["flat_runs"] == 2 and p.info["run_b"] == 32, p.describe()
    err, msg, cnt = emu.run(p, counts=True)
    assert err == 0, msg
    assert cnt.min() == 1 and cnt.max() == 1


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_flat_stream_walk_matches_oracle(dtype):
    """Kernel S walking B flat (rows whose length is not a multiple of the
    vector width, or any compact B when forced): every element written once
    and bit-exact, vectors that cross into the next row, a partial last
    vector, narrower widths for misaligned B pointers."""
    rng = np.random.default_rng(1705)
    seen = 0
    for size_a, perm in [((63, 5, 7), (0, 2, 1)), ((17, 3, 4, 5), (0, 3, 1, 2)),
                         ((75, 10, 11), (0, 2, 1)), ((33, 7, 3, 2), (0, 2, 3, 1)),
                         ((64, 5, 6), (0, 2, 1)), ((21, 9), (0, 1)), ((19, 4, 3), (0, 2, 1)),
                         ((42, 5, 3, 7), (0, 3, 1, 2))]:
        for knobs in (dict(), dict(flat_runs=1)):
            for alpha, beta in ((1.0, 0.0), (1.5, 0.0), (-0.3, 1.25)):
                p = emu.plan(perm, size_a, alpha, beta, dtype, **knobs)
                if p.info["kernel"] != "stream" or not p.info["flat_runs"]:
                    continue
                seen += 1
                for vb in (0, 2, 1):
                    _check(p, size_a, perm, alpha, beta, dtype, rng, vb=vb)
    assert seen >= 12


def test_sheared_whole_short_index_matches_oracle():
    """Sheared tiles holding a short stride-1 A index whole (B runs of two
    lines), with ragged B-run chunks, in both update modes."""
    rng = np.random.default_rng(66)
    for size_a, perm, dtype in [((66, 3000), (1, 0), "f32"), ((69, 90, 70), (1, 2, 0), "f32")]:
        p = emu.plan(perm, size_a, 1.0, 0.0, dtype)
        assert p.info["shear"] > 0 and p.info["run_a"] == size_a[0], p.describe()
        _check(p, size_a, perm, 1.0, 0.0, dtype, rng)
        q = emu.plan(perm, size_a, -0.3, 1.25, dtype, shear=1)
        _check(q, size_a, perm, -0.3, 1.25, dtype, rng)
    # fp64 takes it at full size only: a dry run of every workgroup
    p = emu.plan((1, 2, 3, 0), (30, 2762, 85, 7), 1.0, 1.0, "f64")
    assert p.info["shear"] > 0 and p.info["run_a"] == 30, p.describe()
    err, msg, cnt = emu.run(p, counts=True)
    assert err == 0, msg
    assert cnt.min() == 1 and cnt.max() == 1


def test_direct_lds_tiles_match_oracle():
    """Tiles fetched straight into LDS (variant kDirect: B only written,
    16-byte A vectors): random shapes with ragged row tails and ragged last
    column chunks, fp32 and fp64, against the oracle, the same plans in the
    register-staged variants, and plans with direct loads switched off."""
    rng = np.random.default_rng(1950)
    seen = 0
    for it in range(800):
        size_a, perm = random_problem(rng, max_dims=5, max_numel=60000,
                                      extents=(2, 3, 4, 8, 12, 16, 17, 32, 33, 64, 65, 96))
        dtype = "f32" if it % 3 else "f64"
        alpha = (1.0, 1.5)[it % 2]
        p = emu.plan(perm, size_a, alpha, 0.0, dtype)
        if not p.info["direct_lds"]:
            continue
        seen += 1
        _check(p, size_a, perm, alpha, 0.0, dtype, rng)
        if it % 3 == 0:
            q = emu.plan(perm, size_a, alpha, 0.0, dtype, direct_lds=2)
            assert not q.info["direct_lds"]
            _check(q, size_a, perm, alpha, 0.0, dtype, rng)
        if it % 3 == 1:  # the register-staged variants on the same plan
            _check(p, size_a, perm, alpha, 0.0, dtype, rng, variant="fast")
            _check(p, size_a, perm, alpha, 0.0, dtype, rng, variant="shifted")
    for size_a, knobs in (((128, 36), dict(run_a=32, run_b=16)), ((128, 64), dict(block=1024)),
                          ((256, 32), dict(max_blocks=7)), ((64, 100), dict(run_a=128, run_b=32))):
        p = emu.plan((1, 0), size_a, 1.5, 0.0, "f32", **knobs)
        assert p.info["direct_lds"], p.describe()
        _check(p, size_a, (1, 0), 1.5, 0.0, "f32", rng)
    assert seen >= 30, seen


@pytest.mark.parametrize("k", [2, 16, 1024])
def test_xcd_groups_match_oracle(k):
    """Tile numbers dealt to the XCDs in groups of k (with and without the
    diagonal rotation, which then advances once per group) still cover every
    tile once: disjoint, sheared, flat, stacked and shared-run tiles, grids
    with and without an incomplete last round of 8k tiles, and kernel S's
    blocks (row and flat walks), against the oracle."""
    rng = np.random.default_rng(77 + k)
    cases = [((1759, 444), (1, 0), {}), ((274, 2280), (1, 0), {}),
             ((427, 110, 3, 35), (3, 2, 1, 0), {}), ((77, 165, 2, 197), (3, 1, 0, 2), {}),
             ((96, 96, 9, 7), (2, 0, 3, 1), {}), ((4, 2, 17, 3, 1225), (2, 1, 3, 0, 4), {}),
             ((24, 20, 16, 24, 18, 5), (5, 2, 0, 4, 1, 3), {}),
             ((33, 17, 65), (2, 0, 1), dict(depth=3)), ((600, 130), (1, 0), dict(max_blocks=7)),
             ((42, 4, 13, 107, 21), (0, 4, 3, 1, 2), {}), ((96, 12, 13, 17), (0, 3, 2, 1), {}),
             ((97, 12, 13, 17), (0, 3, 2, 1), dict(flat_runs=2))]
    for size_a, perm, knobs in cases:
        for beta, order in ((0.0, 0), (1.0, 1), (0.5, 2)):
            kw = dict(knobs, xcd_group=k)
            p0 = emu.plan(perm, size_a, 1.5, beta, "f32", **kw)
            if order and p0.info["kernel"] == "tile":
                kw["tile_order"] = order
            p = emu.plan(perm, size_a, 1.5, beta, "f32", **kw)
            if p.info["kernel"] not in ("tile", "stream"):
                continue
            assert p.info["xcd_group"] == k, p.describe()
            _check(p, size_a, perm, 1.5, beta, "f32", rng)
