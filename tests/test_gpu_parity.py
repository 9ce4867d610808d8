"""Parity of the HIP path with the CPU oracle, element by element, on an
MI355X.  Every call goes through the C ABI (paper_1704_04374_amd.hptt).

Bar: bit-exact.  The kernels and the oracle both compute
fl(fl(alpha*a) + fl(beta*b)) in the tensor dtype with no fused multiply-add
(and a raw copy for alpha = 1, beta = 0), so no rounding difference is
expected; the relative-error bound 2^-22 (fp32) / 2^-51 (fp64) is what the
results must meet at the very least, and is reported on failure.
"""
from __future__ import annotations

import itertools

import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_1704_04374_amd import hptt
from paper_1704_04374_amd.workloads import (NUMPY_DTYPE, SUBTENSOR_WORKLOADS, WORKLOADS, inputs,
                                            random_problem, uniform)

pytestmark = pytest.mark.gpu

REL_BOUND = {"f32": 2.0 ** -22, "f64": 2.0 ** -51}
TORCH = {"f32": torch.float32, "f64": torch.float64}


def _say(msg):
    print(msg, flush=True)


def _assert_parity(got: np.ndarray, want: np.ndarray, dtype: str, what: str):
    if np.array_equal(got, want, equal_nan=True):
        return
    bad = np.flatnonzero(~((got == want) | (np.isnan(got) & np.isnan(want))))
    with np.errstate(all="ignore"):
        rel = np.abs(got[bad].astype(np.float64) - want[bad]) / np.maximum(
            np.abs(want[bad].astype(np.float64)), np.finfo(np.float64).tiny)
    raise AssertionError(f"{what}: {bad.size} elements differ, first at {bad[0]} "
                         f"(got {got[bad[0]]!r}, want {want[bad[0]]!r}), max rel err "
                         f"{rel.max():.3e} (bound {REL_BOUND[dtype]:.3e})")


def _rand(rng, n, dtype):
    return (rng.integers(-(1 << 20), 1 << 20, size=n) / float(1 << 20)).astype(NUMPY_DTYPE[dtype])


def _run_case(size_a, perm, alpha, beta, dtype, rng, **knobs):
    p = hptt.create_plan(perm, size_a, alpha, beta, dtype, **knobs)
    n = p.numel
    A = _rand(rng, n, dtype)
    B0 = _rand(rng, n, dtype) if beta != 0 else np.full(n, np.nan, NUMPY_DTYPE[dtype])
    want = orc.transpose(A, size_a, perm, alpha, beta, B0 if beta != 0 else None)
    dA = torch.from_numpy(A).cuda()
    dB = torch.from_numpy(B0).cuda()
    p.exec(dA, dB)
    torch.cuda.synchronize()
    _assert_parity(dB.cpu().numpy(), want, dtype, p.describe())
    return p


@pytest.mark.parametrize("w", WORKLOADS, ids=lambda w: w.name)
def test_workload_full_size(w):
    """Each named workload at its full size, in the launch configuration the
    benchmark times, against the whole oracle result."""
    _say(f"[parity] {w.describe()}")
    A, B0 = inputs(w)
    if B0 is None:
        B0 = torch.full_like(A, float("nan"))   # beta = 0: B must be fully overwritten
    want = orc.transpose(A.numpy(), w.size_a, w.perm, w.alpha, w.beta,
                         B0.numpy() if w.beta != 0 else None)
    p = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype)
    dA, dB = A.cuda(), B0.cuda()
    p.exec(dA, dB)
    torch.cuda.synchronize()
    got = dB.cpu().numpy()
    _assert_parity(got, want, w.dtype, p.describe())
    # one-by-one samples from the oracle agree too (first, last, random)
    rng = np.random.default_rng(w.seed_a)
    offs = np.concatenate([[0, w.numel - 1], rng.integers(0, w.numel, 2000)])
    samp = orc.sample(A.numpy(), w.size_a, w.perm, w.alpha, w.beta,
                      B0.numpy() if w.beta != 0 else None, offs)
    _assert_parity(got[offs], samp, w.dtype, "sampled " + p.describe())


def test_random_sweep():
    """Seeded sweep of small odd shapes: rank 1..6, extents with tails, both
    dtypes, several alpha and beta, every kernel class the plan builder
    chooses (the generic kernel only where forced, in test_forced_variants)."""
    rng = np.random.default_rng(4374)
    seen = set()
    alphas, betas = (1.0, 1.5, -0.3), (0.0, 1.0, 0.5, -1.25)
    for it in range(160):
        size_a, perm = random_problem(rng, max_dims=6, max_numel=1 << 18)
        dtype = ("f32", "f64")[it % 2]
        alpha, beta = alphas[it % 3], betas[(it // 3) % 4]
        p = _run_case(size_a, perm, alpha, beta, dtype, rng)
        seen.add(p.info["kernel"] + ("+shared" if p.info["shared_runs"] else ""))
    assert {"tile", "tile+shared", "axpby", "stream"} <= seen


@pytest.mark.parametrize("w", [w for w in WORKLOADS if w.beta == 0], ids=lambda w: w.name)
def test_workload_full_size_register_staged(w):
    """The named workloads whose tiles are fetched straight into LDS, at full
    size with the register-staged load phase instead (direct_lds = 2)."""
    _say(f"[parity] {w.describe()} direct_lds=2")
    A, _ = inputs(w)
    B = torch.full_like(A, float("nan"))
    want = orc.transpose(A.numpy(), w.size_a, w.perm, w.alpha, w.beta, None)
    p = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype, direct_lds=2)
    assert not p.info["direct_lds"]
    dA, dB = A.cuda(), B.cuda()
    p.exec(dA, dB)
    torch.cuda.synchronize()
    _assert_parity(dB.cpu().numpy(), want, w.dtype, p.describe())


@pytest.mark.parametrize("knobs", [dict(kernel="generic"), dict(run_a=8, run_b=8),
                                   dict(run_a=3, run_b=5), dict(max_blocks=7),
                                   dict(max_vec=1), dict(store_hint=1, load_hint=1), dict(lds_pad=-1),
                                   dict(tile_order=1), dict(tile_order=3), dict(run_a=512, run_b=8),
                                   dict(row_passes=3), dict(row_passes=2, max_blocks=5),
                                   dict(run_a=64, run_b=64, max_blocks=5),
                                   dict(exact_runs=1, run_a=6, run_b=10),
                                   dict(block=1024), dict(block=1024, run_a=64, run_b=64),
                                   dict(block=1024, max_blocks=5), dict(tile_order=4),
                                   dict(skew=3), dict(store_hint=2, load_hint=2),
                                   dict(grid_order=2), dict(grid_order=3), dict(direct_lds=2),
                                   dict(block=1024, run_a=128, run_b=32), dict(xcd_group=16),
                                   dict(xcd_group=2, max_blocks=5),
                                   dict(xcd_group=1024, tile_order=1)],
                         ids=lambda k: ",".join(f"{a}={b}" for a, b in k.items()))
def test_forced_variants(knobs):
    rng = np.random.default_rng(99)
    for size_a, perm in [((65, 65), (1, 0)), ((33, 17, 5), (2, 0, 1)),
                         ((24, 20, 16, 5, 3), (4, 2, 0, 3, 1)), ((3, 2, 64, 9, 32), (4, 2, 0, 3, 1))]:
        for dtype, (alpha, beta) in (("f32", (1.0, 0.0)), ("f64", (1.5, -0.5))):
            _run_case(size_a, perm, alpha, beta, dtype, rng, **knobs)


@pytest.mark.parametrize("name,knobs", [
    ("transpose6d_24x20x16x24x18x20_f32", dict(exact_runs=1, run_a=96, run_b=160, block=1024)),
    ("transpose6d_24x20x16x24x18x20_f32", dict(exact_runs=1, run_a=96, run_b=320, block=1024)),
    ("transpose5d_3x2x640x480x96_f32", dict(exact_runs=1, run_a=192, run_b=96, block=1024)),
    ("transpose2d_8192x8192_f32", dict(block=1024, tile_order=4)),
    ("transpose2d_8192x8192_f32", dict(block=1024, run_a=128, run_b=32)),
    ("transpose2d_8192x8192_f32", dict(xcd_group=16)),
    ("transpose5d_3x2x640x480x96_f32", dict(xcd_group=8, tile_order=1))],
    ids=lambda x: x if isinstance(x, str) else ",".join(f"{a}={b}" for a, b in x.items()))
def test_large_tiles_full_size(name, knobs):
    """1024-thread workgroups and tiles above 64 KiB of LDS (register-staged
    and, for the 2-D 128x32 tile, fetched straight into LDS), and tiles dealt
    to the XCDs in groups, at full size, against the whole oracle result."""
    from paper_1704_04374_amd.workloads import BY_NAME
    w = BY_NAME[name]
    _say(f"[parity] {w.describe()} {knobs}")
    A, B0 = inputs(w)
    if B0 is None:
        B0 = torch.full_like(A, float("nan"))
    want = orc.transpose(A.numpy(), w.size_a, w.perm, w.alpha, w.beta,
                         B0.numpy() if w.beta != 0 else None)
    p = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype, **knobs)
    if "block" in knobs:
        assert p.info["block"] == 1024
    if "xcd_group" in knobs:
        assert p.info["xcd_group"] == knobs["xcd_group"]
    dA, dB = A.cuda(), B0.cuda()
    p.exec(dA, dB)
    torch.cuda.synchronize()
    _assert_parity(dB.cpu().numpy(), want, w.dtype, p.describe())


def test_sheared_b_runs():
    """B runs sheared onto 128-byte lines, small (forced) and at sweep size,
    including tensors that start off a line."""
    rng = np.random.default_rng(41)
    sheared = 0
    for size_a, perm in [((397, 125), (1, 0)), ((153, 10, 325), (2, 0, 1)),
                         ((65, 33, 129), (2, 0, 1))]:
        for dtype, (alpha, beta) in (("f32", (1.0, 0.0)), ("f64", (1.5, -0.5)),
                                     ("f32", (2.0, 0.5))):
            p = _run_case(size_a, perm, alpha, beta, dtype, rng, shear=1)
            sheared += p.info["shear"] > 0
    assert sheared >= 6
    for size_a, perm in [((39792, 1257), (1, 0)), ((1538, 10, 3251), (2, 0, 1))]:
        p = _run_case(size_a, perm, 1.0, 0.0, "f32", rng)
        assert p.info["shear"] == 31
    # tensors one and three elements past a line
    p = hptt.create_plan((1, 0), (397, 125), 1.5, 0.5, "f64", shear=1)
    for off in (1, 3):
        n = p.numel
        A = _rand(rng, n, "f64")
        B0 = _rand(rng, n, "f64")
        want = orc.transpose(A, (397, 125), (1, 0), 1.5, 0.5, B0)
        dA = torch.zeros(n + 8, dtype=torch.float64, device="cuda")
        dB = torch.zeros(n + 8, dtype=torch.float64, device="cuda")
        dA[off:off + n] = torch.from_numpy(A).cuda()
        dB[off:off + n] = torch.from_numpy(B0).cuda()
        p.exec(dA[off:off + n], dB[off:off + n])
        torch.cuda.synchronize()
        got = dB.cpu().numpy()
        _assert_parity(got[off:off + n], want, "f64", f"offset {off}: {p.describe()}")
        assert np.all(got[:off] == 0) and np.all(got[off + n:] == 0)


def test_flat_b_runs():
    """B runs cut in whole lines from the flattened range of two or more B
    indices (row tables rebuilt per tile): small forced cases with partial
    last chunks, tensors that start off the vector grid, and the 6-D fp32
    workload's plan on a smaller grid."""
    rng = np.random.default_rng(43)
    flat = 0
    for size_a, perm in [((24, 6, 16, 20), (3, 2, 0, 1)), ((10, 3, 5, 7), (3, 2, 1, 0)),
                         ((33, 2, 9, 11), (2, 3, 0, 1)), ((5, 40, 3, 6, 7), (4, 3, 2, 0, 1)),
                         ((24, 20, 16, 3, 2, 20), (5, 2, 0, 4, 1, 3))]:
        for knobs in (dict(), dict(run_b=8), dict(run_a=16, run_b=8)):
            for dtype, (alpha, beta) in (("f32", (1.0, 0.0)), ("f64", (1.5, -0.5)),
                                         ("f32", (2.0, 0.5))):
                p = _run_case(size_a, perm, alpha, beta, dtype, rng, flat_runs=1, **knobs)
                flat += p.info["flat_runs"] > 0
    assert flat >= 12
    p = hptt.create_plan((5, 2, 0, 4, 1, 3), (24, 20, 16, 3, 2, 20), 1.5, 0.5, "f32")
    assert p.info["flat_runs"] == 2, p.describe()
    for off in (1, 3):
        n = p.numel
        A = _rand(rng, n, "f32")
        B0 = _rand(rng, n, "f32")
        want = orc.transpose(A, (24, 20, 16, 3, 2, 20), (5, 2, 0, 4, 1, 3), 1.5, 0.5, B0)
        dA = torch.zeros(n + 8, dtype=torch.float32, device="cuda")
        dB = torch.zeros(n + 8, dtype=torch.float32, device="cuda")
        dA[off:off + n] = torch.from_numpy(A).cuda()
        dB[off:off + n] = torch.from_numpy(B0).cuda()
        p.exec(dA[off:off + n], dB[off:off + n])
        torch.cuda.synchronize()
        got = dB.cpu().numpy()
        _assert_parity(got[off:off + n], want, "f32", f"offset {off}: {p.describe()}")
        assert np.all(got[:off] == 0) and np.all(got[off + n:] == 0)


def test_shared_runs():
    """Tiles whose A run and B run share indices (a B stride-1 extent of 2, a
    short kept stride-1 index, a small block permuted inside itself), forced,
    over every update mode, both dtypes and ragged chunks, and on tensors
    that start off the vector grid (runs shifted onto it)."""
    rng = np.random.default_rng(57)
    shapes = [((12, 3, 2, 23, 13), (2, 1, 4, 3, 0)), ((184, 2, 1350), (1, 0, 2)),
              ((2925, 12, 2, 7), (2, 0, 3, 1)), ((125, 2, 5, 39), (2, 0, 3, 1)),
              ((70, 5, 98), (1, 0, 2)), ((4, 2, 17, 3, 122), (2, 1, 3, 0, 4)),
              ((2, 44, 570), (1, 0, 2)), ((71, 2, 2, 176), (2, 0, 3, 1)),
              ((2, 2625, 4, 23), (1, 3, 0, 2)), ((22, 6, 2, 82, 8, 3), (4, 1, 5, 3, 0, 2)),
              ((32678, 15), (1, 0)), ((26, 15, 11, 2, 58), (3, 2, 0, 4, 1)),
              ((2, 6025, 41), (0, 2, 1)), ((2, 454, 19, 27, 10), (0, 3, 2, 1, 4)),
              ((4, 2, 82, 15, 7, 7), (0, 4, 2, 1, 5, 3)), ((14, 35820), (1, 0))]
    modes = [(1.0, 0.0), (1.5, 0.0), (2.0, 0.5), (-0.3, 1.25)]
    seen = 0
    for i, (size_a, perm) in enumerate(shapes):
        dtype = ("f32", "f64")[i % 2]
        alpha, beta = modes[i % len(modes)]
        _say(f"[parity] shared runs {size_a} {perm} {dtype} {alpha} {beta}")
        p = _run_case(size_a, perm, alpha, beta, dtype, rng, shared_runs=1)
        seen += p.info["shared_runs"] > 0
    assert seen == len(shapes)
    for (size_a, perm), dtype, off in itertools.product(
            [((184, 2, 1350), (1, 0, 2)), ((2, 6025, 41), (0, 2, 1))], ("f32", "f64"), (1, 3)):
        p = hptt.create_plan(perm, size_a, 1.5, 0.5, dtype, shared_runs=1)
        n = p.numel
        A = _rand(rng, n, dtype)
        B0 = _rand(rng, n, dtype)
        want = orc.transpose(A, size_a, perm, 1.5, 0.5, B0)
        bufA = torch.zeros(n + 8, dtype=TORCH[dtype], device="cuda")
        bufB = torch.zeros(n + 8, dtype=TORCH[dtype], device="cuda")
        dA, dB = bufA[off:off + n], bufB[off:off + n]
        dA.copy_(torch.from_numpy(A))
        dB.copy_(torch.from_numpy(B0))
        p.exec(dA, dB)
        torch.cuda.synchronize()
        _assert_parity(dB.cpu().numpy(), want, dtype, f"offset {off}: {p.describe()}")
        assert bufB[:off].abs().sum().item() == 0 and bufB[off + n:].abs().sum().item() == 0


def test_stream_kernel_variants():
    rng = np.random.default_rng(5)
    for size_a, perm in [((96, 7, 9, 5), (0, 3, 2, 1)), ((33, 8, 8), (0, 2, 1)),
                         ((16, 5, 6), (0, 2, 1))]:
        for knobs in (dict(), dict(max_vec=1), dict(max_blocks=3)):
            _run_case(size_a, perm, 2.0, 0.5, "f64", rng, kernel="stream", **knobs)
            _run_case(size_a, perm, 1.0, 0.0, "f32", rng, kernel="stream", **knobs)


def test_flat_stream_walk():
    """Kernel S walking B flat (odd fp32 rows by default, any compact B
    when forced): vectors that cross rows, a partial last vector, capped
    grids, and B pointers 1 to 3 elements off the 16-byte grid."""
    rng = np.random.default_rng(55)
    flat = 0
    for size_a, perm in [((63, 5, 7), (0, 2, 1)), ((17, 3, 4, 5), (0, 3, 1, 2)),
                         ((75, 10, 11), (0, 2, 1)), ((19, 4, 3), (0, 2, 1)),
                         ((42, 5, 3, 7), (0, 3, 1, 2))]:
        for knobs in (dict(), dict(flat_runs=1), dict(max_blocks=3)):
            for dtype, (alpha, beta) in (("f32", (1.0, 0.0)), ("f32", (2.0, 0.5)),
                                         ("f64", (1.5, -0.5))):
                p = _run_case(size_a, perm, alpha, beta, dtype, rng, **knobs)
                flat += p.info["kernel"] == "stream" and p.info["flat_runs"] == 1
    assert flat >= 20
    size_a, perm = (63, 5, 7), (0, 2, 1)
    p = hptt.create_plan(perm, size_a, 1.5, 0.5, "f32")
    assert p.info["flat_runs"] == 1, p.describe()
    for off in (1, 2, 3):
        n = p.numel
        A = _rand(rng, n, "f32")
        B0 = _rand(rng, n, "f32")
        want = orc.transpose(A, size_a, perm, 1.5, 0.5, B0)
        dA = torch.zeros(n + 8, dtype=torch.float32, device="cuda")
        dB = torch.zeros(n + 8, dtype=torch.float32, device="cuda")
        dA[off:off + n] = torch.from_numpy(A).cuda()
        dB[4 - off:4 - off + n] = torch.from_numpy(B0).cuda()
        p.exec(dA[off:off + n], dB[4 - off:4 - off + n])
        torch.cuda.synchronize()
        got = dB.cpu().numpy()
        _assert_parity(got[4 - off:4 - off + n], want, "f32", f"offset {off}: {p.describe()}")
        assert np.all(got[:4 - off] == 0) and np.all(got[4 - off + n:] == 0)


def test_misaligned_pointers_fall_back():
    """Tensors starting one element past a 16-byte boundary take narrower
    vector accesses and stay correct."""
    rng = np.random.default_rng(3)
    for (size_a, perm, dtype), pipe in itertools.product(
            [((64, 64), (1, 0), "f32"), ((3, 2, 64, 8, 32), (4, 2, 0, 3, 1), "f32"),
             ((96, 6, 7), (0, 2, 1), "f64"), ((1000,), (0,), "f32")], (1, 2)):
        p = hptt.create_plan(perm, size_a, 1.5, 0.5, dtype, tile_order=pipe)
        n = p.numel
        A = _rand(rng, n, dtype)
        B0 = _rand(rng, n, dtype)
        want = orc.transpose(A, size_a, perm, 1.5, 0.5, B0)
        bufA = torch.zeros(n + 1, dtype=TORCH[dtype], device="cuda")
        bufB = torch.zeros(n + 3, dtype=TORCH[dtype], device="cuda")
        dA, dB = bufA[1:], bufB[3:3 + n]
        dA.copy_(torch.from_numpy(A))
        dB.copy_(torch.from_numpy(B0))
        p.exec(dA, dB)
        torch.cuda.synchronize()
        _assert_parity(dB.cpu().numpy(), want, dtype, "misaligned " + p.describe())
        assert bufB[:3].abs().sum().item() == 0      # nothing written before B


def test_overlap_rejected_and_nothing_written():
    p = hptt.create_plan((1, 0), (64, 64))
    buf = torch.zeros(64 * 64 + 64, device="cuda")
    with pytest.raises(hptt.HpttError) as e:
        p.exec(buf[:4096].data_ptr(), buf[64:].data_ptr())
    assert e.value.status == 3
    torch.cuda.synchronize()
    assert buf.abs().sum().item() == 0


def test_load_kernels_then_exec():
    """hptt_load_kernels loads every code object without launching anything
    (twice: a second call is a no-op) and leaves every kernel class usable."""
    hptt.load_kernels()
    hptt.load_kernels()
    rng = np.random.default_rng(11)
    for size_a, perm, beta, dtype in [((64, 48, 5), (1, 0, 2), 0.0, "f32"),
                                      ((65, 33, 17), (2, 0, 1), 0.5, "f64"),
                                      ((33, 7, 5), (0, 2, 1), 1.0, "f32")]:
        _run_case(size_a, perm, 1.5, beta, dtype, rng)


def test_zero_size_is_noop():
    p = hptt.create_plan((2, 1, 0), (4, 0, 3))
    assert p.info["kernel"] == "none"
    p.exec(0, 0)
    torch.cuda.synchronize()


def test_alpha_zero_beta_one_keeps_b():
    """The non-destructive autotuning setting of Section 3.1: alpha = 0,
    beta = 1 rewrites B with its own value (A finite, footnote 5)."""
    rng = np.random.default_rng(8)
    for size_a, perm in [((128, 96), (1, 0)), ((24, 20, 16), (2, 0, 1))]:
        A = torch.from_numpy(_rand(rng, int(np.prod(size_a)), "f32")).cuda()
        B0 = torch.from_numpy(_rand(rng, A.numel(), "f32") + np.float32(0.5)).cuda()
        B = B0.clone()
        hptt.create_plan(perm, size_a, 0.0, 1.0).exec(A, B)
        torch.cuda.synchronize()
        assert torch.equal(B, B0)


def test_streams_and_plan_reuse():
    """One plan executed on two streams and repeatedly; results independent."""
    rng = np.random.default_rng(21)
    size_a, perm = (256, 96, 8), (1, 2, 0)
    p = hptt.create_plan(perm, size_a, 1.0, 0.0)
    n = p.numel
    As = [_rand(rng, n, "f32") for _ in range(2)]
    wants = [orc.transpose(a, size_a, perm) for a in As]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    dA = [torch.from_numpy(a).cuda() for a in As]
    dB = [torch.empty_like(x) for x in dA]
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            p.exec(dA[0], dB[0])
        with torch.cuda.stream(s2):
            p.exec(dA[1], dB[1])
    torch.cuda.synchronize()
    for b, w in zip(dB, wants):
        _assert_parity(b.cpu().numpy(), w, "f32", p.describe())


def test_graph_capture_replays():
    """hptt_exec captured into a HIP graph and replayed four times, with eager
    work and synchronisations between the replays: every replay matches the
    oracle (tile, shared-run, sheared, stream and generic plans; with beta !=
    0, B is reset eagerly before each replay, outside the graph)."""
    rng = np.random.default_rng(41)
    cases = [((256, 96, 8), (1, 2, 0), 1.5, 0.0, "f32", {}),
             ((12, 3, 2, 93, 33), (2, 1, 4, 3, 0), 1.5, 0.0, "f32", {}),
             ((66, 7576), (1, 0), 1.0, 1.0, "f32", dict(shear=1)),
             ((96, 40, 6), (0, 2, 1), 2.0, 0.5, "f64", {}),
             ((17, 5, 33), (2, 0, 1), 1.0, 1.0, "f32", dict(kernel="generic"))]
    for size_a, perm, alpha, beta, dtype, knobs in cases:
        p = hptt.create_plan(perm, size_a, alpha, beta, dtype, **knobs)
        _say(f"graph: {p.describe()}")
        n = p.numel
        A = _rand(rng, n, dtype)
        B0 = _rand(rng, n, dtype) if beta != 0 else np.full(n, np.nan, NUMPY_DTYPE[dtype])
        want = orc.transpose(A, size_a, perm, alpha, beta, B0 if beta != 0 else None)
        dA = torch.from_numpy(A).cuda()
        dB0 = torch.from_numpy(B0).cuda()
        dB = dB0.clone()
        p.exec(dA, dB)  # eager run first: the kernel is loaded before capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            p.exec(dA, dB)
        for rep in range(4):
            dB.copy_(dB0)
            junk = torch.empty(1 << 20, device="cuda").uniform_()  # eager work between replays
            g.replay()
            torch.cuda.synchronize()
            _assert_parity(dB.cpu().numpy(), want, dtype, f"replay {rep}: {p.describe()}")
            del junk


def test_inverse_round_trip_on_gpu():
    """Pi then Pi^-1 returns A bit for bit on the device."""
    rng = np.random.default_rng(31)
    for size_a, perm in [((24, 20, 16, 24, 3), (4, 2, 0, 3, 1)), ((130, 70), (1, 0))]:
        inv = [0] * len(perm)
        for k, q in enumerate(perm):
            inv[q] = k
        size_b = tuple(size_a[q] for q in perm)
        A = torch.from_numpy(_rand(rng, int(np.prod(size_a)), "f64")).cuda()
        B = torch.empty_like(A)
        C = torch.empty_like(A)
        hptt.create_plan(perm, size_a, dtype="f64").exec(A, B)
        hptt.create_plan(inv, size_b, dtype="f64").exec(B, C)
        torch.cuda.synchronize()
        assert torch.equal(A, C)


def test_yardsticks():
    n = 1 << 20
    x = torch.rand(n, device="cuda")
    y = torch.rand(n, device="cuda")
    z = torch.empty_like(x)
    hptt.yardstick_copy(x, z, n * 4)
    torch.cuda.synchronize()
    assert torch.equal(x, z)
    y0 = y.clone()
    hptt.yardstick_axpby("f32", 2.0, x, 0.5, y, n)
    torch.cuda.synchronize()
    assert torch.equal(y.cpu(), 2.0 * x.cpu() + 0.5 * y0.cpu())
    hptt.yardstick_fill(z, n * 4, 0)
    torch.cuda.synchronize()
    assert z.abs().sum().item() == 0


# --------------------------------------------------------------------------
# Sub-tensors with outer sizes (Section 3.1, Fig. 3)
# --------------------------------------------------------------------------

def _fortran_offset(index, outer):
    off, stride = 0, 1
    for i, o in zip(index, outer):
        off += int(i) * stride
        stride *= int(o)
    return off


def _run_outer(size_a, perm, outer_a, outer_b, start_a, start_b, alpha, beta, dtype, rng,
               **knobs):
    p = hptt.create_plan(perm, size_a, alpha, beta, dtype, outer_size_a=outer_a,
                         outer_size_b=outer_b, **knobs)
    npd = NUMPY_DTYPE[dtype]
    PA = _rand(rng, int(np.prod(outer_a)), dtype)
    PB = _rand(rng, int(np.prod(outer_b)), dtype)
    oa, ob = _fortran_offset(start_a, outer_a), _fortran_offset(start_b, outer_b)
    want = np.concatenate([PB[:ob], orc.transpose_outer(PA[oa:], size_a, perm, outer_a, outer_b,
                                                        alpha, beta, PB[ob:])])
    dA = torch.from_numpy(PA).cuda()
    dB = torch.from_numpy(PB).cuda()
    p.exec(dA[oa:], dB[ob:])
    torch.cuda.synchronize()
    _assert_parity(dB.cpu().numpy(), want.astype(npd), dtype, "outer " + p.describe())
    return p


def test_fig3b_sub_tensor_on_gpu():
    """Fig. 3b: the 8x16x16 sub-tensor of a 16x32x32 tensor, compacted."""
    rng = np.random.default_rng(3)
    _run_outer((8, 16, 16), (2, 1, 0), (16, 32, 32), (16, 16, 8), (0, 0, 0), (0, 0, 0),
               1.0, 0.0, "f32", rng)
    # the same sub-tensor taken from the middle of A, and scattered back
    _run_outer((8, 16, 16), (2, 1, 0), (16, 32, 32), (16, 32, 16), (5, 9, 11), (0, 7, 3),
               1.5, 0.5, "f64", rng)


@pytest.mark.parametrize("knobs", [dict(), dict(kernel="generic"), dict(run_a=8, run_b=8)],
                         ids=["default", "generic", "small_tiles"])
def test_sub_tensors_random(knobs):
    rng = np.random.default_rng(77)
    kinds = set()
    for it in range(60):
        n = int(rng.integers(1, 6))
        size_a = tuple(int(x) for x in rng.choice([1, 2, 3, 5, 8, 17, 33, 64, 65], size=n))
        if np.prod(size_a) > (1 << 17):
            continue
        perm = tuple(int(p) for p in rng.permutation(n))
        size_b = tuple(size_a[p] for p in perm)
        outer_a = tuple(s + int(rng.choice([0, 0, 1, 3, 8])) for s in size_a)
        outer_b = tuple(s + int(rng.choice([0, 0, 1, 3, 8])) for s in size_b)
        start_a = tuple(int(rng.integers(0, o - s + 1)) for s, o in zip(size_a, outer_a))
        start_b = tuple(int(rng.integers(0, o - s + 1)) for s, o in zip(size_b, outer_b))
        dtype = ("f32", "f64")[it % 2]
        alpha, beta = ((1.0, 0.0), (1.5, 0.0), (-0.3, 1.25), (2.0, 0.5))[it % 4]
        p = _run_outer(size_a, perm, outer_a, outer_b, start_a, start_b, alpha, beta, dtype,
                       rng, **knobs)
        kinds.add(p.info["kernel"])
    if not knobs:
        assert {"tile", "generic"} <= kinds


@pytest.mark.parametrize("w", SUBTENSOR_WORKLOADS, ids=lambda w: w.name)
def test_sub_tensor_workload_full_size(w):
    """The transpose-and-compact and transpose-and-scatter workloads the
    benchmark times (halves of an 8192 x 8192 matrix, Fig. 3), with the plan
    the benchmark builds, compared whole against the oracle: every element of
    the enclosing B, including those outside the sub-tensor, which must keep
    their prior (NaN) bits."""
    _say(w.describe())
    PA = uniform(w.parent_numel_a, w.dtype, w.seed_a).numpy()
    PB = np.full(w.parent_numel_b, np.nan, dtype=NUMPY_DTYPE[w.dtype])
    oa, ob = w.offset_a, w.offset_b
    outer_a = w.outer_a or w.size_a
    outer_b = w.outer_b or w.size_b
    p = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype, outer_size_a=w.outer_a,
                         outer_size_b=w.outer_b)
    want = np.concatenate([PB[:ob], orc.transpose_outer(PA[oa:], w.size_a, w.perm, outer_a,
                                                        outer_b, w.alpha, w.beta, PB[ob:])])
    dA = torch.from_numpy(PA).cuda()
    dB = torch.from_numpy(PB).cuda()
    p.exec(dA[oa:], dB[ob:])
    torch.cuda.synchronize()
    got = dB.cpu().numpy()
    assert got.tobytes() == want.tobytes(), p.describe()
    # the region outside the sub-tensor is untouched, and nothing inside is NaN
    inside = np.zeros(w.parent_numel_b, dtype=bool)
    inside[ob:] = ~np.isnan(want[ob:])
    assert np.isnan(got[~inside]).all() and not np.isnan(got[inside]).any()
    assert inside.sum() == w.numel


# --------------------------------------------------------------------------
# Beyond 32-bit element counts, and ranks up to 16
# --------------------------------------------------------------------------

def test_above_2_31_elements():
    """A 46341 x 46341 fp32 transposition (2,147,488,281 elements, 8.6 GB per
    tensor): the tile kernel's 64-bit offset variant.  With alpha = 1.5,
    beta = -0.5 on a random prior B, then alpha = 1, beta = 0 on a NaN-filled
    B: sampled elements (the first and last included) against the oracle
    computed one by one, and no NaN left anywhere in B."""
    size, perm = (46341, 46341), (1, 0)
    n = size[0] * size[1]
    _say(f"[parity] {size} perm {perm}: {n} elements")
    g = torch.Generator(device="cuda").manual_seed(31)
    dA = torch.rand(n, device="cuda", generator=g) * 2 - 1
    dB = torch.rand(n, device="cuda", generator=g) * 2 - 1
    hA, hB0 = dA.cpu().numpy(), dB.cpu().numpy()
    rng = np.random.default_rng(31)
    offs = np.concatenate([[0, 1, n - 2, n - 1, 2 ** 31 - 1, 2 ** 31, 2 ** 31 + 1],
                           rng.integers(0, n, 6000)])
    toffs = torch.from_numpy(offs).cuda()
    for alpha, beta in ((1.5, -0.5), (1.0, 0.0)):
        p = hptt.create_plan(perm, size, alpha, beta, "f32")
        if beta == 0:
            dB.fill_(float("nan"))
        p.exec(dA, dB)
        torch.cuda.synchronize()
        got = dB[toffs].cpu().numpy()
        want = orc.sample(hA, size, perm, alpha, beta, hB0 if beta != 0 else None, offs)
        assert got.tobytes() == want.tobytes(), p.describe()
        assert not bool(torch.isnan(dB).any()), p.describe()
    del dA, dB


def test_high_ranks():
    """Ranks 7 to 16 (extents 2 and 3, fusion and dropped extent-1 indices
    included), both dtypes, whole results against the oracle."""
    rng = np.random.default_rng(16)
    for n in range(7, 17):
        for it in range(3):
            size = [int(x) for x in rng.choice([1, 2, 2, 3], size=n)]
            while int(np.prod(size)) > (1 << 17):
                size[int(rng.integers(0, n))] = 2
            perm = tuple(int(x) for x in rng.permutation(n))
            dtype = ("f32", "f64")[it % 2]
            alpha, beta = ((1.0, 0.0), (-0.375, 1.25), (2.0, 0.5))[it]
            p = _run_case(tuple(size), perm, alpha, beta, dtype, rng)
            assert p.info["numel"] == int(np.prod(size))


def test_stream_slabs_above_2_32_items():
    """The stride-1-kept walk with more than 2^32 vectors: 64 x 4096 x 16385
    fp32 (2^32 + 2^18 elements, 17 GB per tensor) on pointers one element off
    the 16-byte grid, so hptt_exec narrows to 1-element vectors and launches
    per slab of the slowest B index.  alpha = -0.5, beta = 1 on a random prior
    B, then alpha = 1, beta = 0 on a NaN-filled B: sampled elements (slab
    edges included) against the oracle computed one by one, no NaN left."""
    size, perm = (64, 4096, 16385), (0, 2, 1)
    n = size[0] * size[1] * size[2]
    _say(f"[parity] {size} perm {perm}: {n} elements, pointers off the vector grid")
    g = torch.Generator(device="cuda").manual_seed(32)
    PA = torch.rand(n + 1, device="cuda", generator=g) * 2 - 1
    PB = torch.rand(n + 1, device="cuda", generator=g) * 2 - 1
    dA, dB = PA[1:], PB[1:]
    hA, hB0 = dA.cpu().numpy(), dB.cpu().numpy()
    rng = np.random.default_rng(32)
    rowsB = size[2] * 64                          # B elements per value of the slowest index
    edges = [0, n - 1, 2 ** 32 - 1, 2 ** 32, 4095 * rowsB - 1, 4095 * rowsB]
    offs = np.concatenate([edges, rng.integers(0, n, 6000)])
    toffs = torch.from_numpy(offs).cuda()
    for alpha, beta in ((-0.5, 1.0), (1.0, 0.0)):
        p = hptt.create_plan(perm, size, alpha, beta, "f32")
        assert p.info["kernel"] == "stream"
        if beta == 0:
            dB.fill_(float("nan"))
        p.exec(dA, dB)
        torch.cuda.synchronize()
        got = dB[toffs].cpu().numpy()
        want = orc.sample(hA, size, perm, alpha, beta, hB0 if beta != 0 else None, offs)
        assert got.tobytes() == want.tobytes(), p.describe()
        assert not bool(torch.isnan(dB).any()), p.describe()
    assert float(PB[0]) == float(PB[0])           # the element before B is untouched (not NaN)
    del PA, PB, dA, dB
