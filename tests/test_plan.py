"""The C ABI and the plan builder, on the CPU (hptt_create_plan makes no HIP
call; hptt_exec's argument checks run before any launch)."""
from __future__ import annotations

import ctypes
import glob
import os
import re

import pytest

from conftest import ROOT, golden
from paper_1704_04374_amd import hptt
from paper_1704_04374_amd.workloads import WORKLOADS, BY_NAME


def _declared_functions(headers=("hptt.h", "hptt_yardstick.h")):
    names = set()
    for name in headers:
        text = open(os.path.join(ROOT, "include", name)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        names.update(re.findall(r"\b(hptt_[a-z0-9_]+)\s*\(", text))
    return names


def test_every_header_is_checked():
    assert sorted(os.path.basename(p) for p in glob.glob(os.path.join(ROOT, "include", "*.h"))) \
        == ["hptt.h", "hptt_contract.h", "hptt_yardstick.h"]


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(hptt.LIB_PATH)
    declared = _declared_functions()
    assert declared, "no declarations found"
    for name in sorted(declared):
        assert hasattr(lib, name), f"{name} declared but not exported"
    assert declared == set(hptt.EXPORTS)


def test_contraction_library_exports_every_declared_symbol():
    from paper_1704_04374_amd import contraction
    lib = ctypes.CDLL(contraction.LIB_PATH)
    declared = _declared_functions(("hptt_contract.h",))
    assert declared
    for name in sorted(declared):
        assert hasattr(lib, name), f"{name} declared but not exported"
    assert declared == set(contraction.EXPORTS)


def test_status_strings():
    lib = hptt.library()
    for code in range(6):
        assert lib.hptt_status_string(code)
    assert lib.hptt_status_string(99) == b"unknown status"


def test_fig1_plan():
    """Fig. 1: B_{i2 i1} <- A_{i1 i2}, A 6x4: a 2-D transpose, nothing to fuse."""
    rows = {r[0]: r[1:] for r in golden("fig1_plan.txt")}
    size_a = tuple(int(x) for x in rows["sizeA"])
    perm = tuple(int(x) for x in rows["perm"])
    info = hptt.create_plan(perm, size_a, shared_runs=2).info
    assert info["size"] == size_a and info["perm"] == perm
    assert info["kernel"] == "tile" and info["dims_a"] == 1 and info["dims_b"] == 1
    # by default so small a problem is one tile whose runs share both indices
    info = hptt.create_plan(perm, size_a).info
    assert info["kernel"] == "tile" and info["shared_runs"] == 2 and info["tiles"] == 1


def test_fn4_fusion():
    """Footnote 4: B_{i2 i3 i1} <- A_{i1 i2 i3} becomes a 2-D problem."""
    rows = {r[0]: r[1:] for r in golden("fn4_fusion.txt")}
    perm = tuple(int(x) for x in rows["perm"])
    fused = tuple(int(x) for x in rows["fused_perm"])
    info = hptt.create_plan(perm, (6, 7, 8)).info
    assert info["ndim"] == 2 and info["size"] == (6, 56) and info["perm"] == fused


@pytest.mark.parametrize("perm,size,fsize,fperm", [
    ((2, 1, 0), (5, 1, 7), (5, 7), (1, 0)),            # extent-1 index dropped
    ((0, 1, 2), (3, 4, 5), (60,), (0,)),               # identity fuses to one index
    ((1, 0), (1, 1), (1,), (0,)),                      # all extents 1
    ((0, 2, 1, 3), (4, 5, 6, 7), (4, 5, 6, 7), (0, 2, 1, 3)),
    ((2, 3, 0, 1), (2, 3, 4, 5), (6, 20), (1, 0)),     # two superindices
    ((3, 0, 1, 2), (2, 3, 4, 5), (24, 5), (1, 0)),
    ((1, 2, 3, 0), (2, 1, 4, 5), (2, 20), (1, 0)),     # extent 1 inside a group
])
def test_fusion_cases(perm, size, fsize, fperm):
    info = hptt.create_plan(perm, size).info
    assert info["size"] == fsize and info["perm"] == fperm


def test_kernel_classes():
    assert hptt.create_plan((0, 1), (5, 7)).info["kernel"] == "axpby"
    assert hptt.create_plan((0, 2, 1), (64, 5, 7)).info["kernel"] == "stream"
    # 12-byte kept rows: a tile whose runs share the kept index, else generic
    info = hptt.create_plan((0, 2, 1), (3, 5, 7)).info
    assert info["kernel"] == "tile" and info["shared_runs"] >= 1
    assert hptt.create_plan((0, 2, 1), (3, 5, 7), shared_runs=2).info["kernel"] == "generic"
    assert hptt.create_plan((1, 0), (5, 7)).info["kernel"] == "tile"
    assert hptt.create_plan((1, 0), (0, 7)).info["kernel"] == "none"


# What the plan builder must decide for each named workload.
EXPECTED = {
    "transpose3d_48x40x32_f32": dict(kernel="tile", size=(1920, 32), perm=(1, 0), run_a=32,
                                     run_b=32, tiles=60),
    "transpose2d_8192x8192_f32": dict(kernel="tile", size=(8192, 8192), perm=(1, 0), run_a=128,
                                      run_b=32, tiles=16384, tile_order=2, hints=3,
                                      grid_order=1, xcd_group=1),
    # flat B runs: one line cut from the 20 x 16 = 320 flattened B positions
    # (10 chunks), A runs of 24 x 4 = 96 elements (3 lines)
    "transpose6d_24x20x16x24x18x20_f32": dict(kernel="tile", size=(24, 20, 16, 24, 18, 20),
                                              perm=(5, 2, 0, 4, 1, 3), run_a=96, run_b=32,
                                              dims_a=2, dims_b=2, tiles=21600, hints=3,
                                              rows_per_pass=32, flat_runs=2,
                                              # outer digits by the sum of their strides: A4
                                              # (B-adjacent) before A3 (A-adjacent)
                                              grid_order=2, xcd_group=1),
    "transpose4d_96x96x96x96_keep1_f64": dict(kernel="stream", size=(96, 96, 96, 96),
                                              perm=(0, 3, 2, 1), run_b=96, vec_a=2, vec_b=2),
    # beta != 0: A-run target of 256 bytes, met by 3 x 2 x 16 = 96 elements (384 B)
    "transpose5d_3x2x640x480x96_f32": dict(kernel="tile", size=(3, 2, 640, 480, 96),
                                           perm=(4, 2, 0, 3, 1), run_a=96, run_b=32, dims_a=3,
                                           dims_b=1, tiles=57600, hints=3, depth=1,
                                           grid_order=1, xcd_group=1),
    # 32-element A runs off the line grid: sheared tiles dealt to the XCDs in
    # groups of 16, grid-digit order
    "xcdgroups2d_2193x22800_f32": dict(kernel="tile", size=(2193, 22800), perm=(1, 0), run_a=32,
                                       run_b=128, shear=31, tile_order=1, xcd_group=16),
}


@pytest.mark.parametrize("name", sorted(EXPECTED))
def test_workload_plans(name):
    w = BY_NAME[name]
    info = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype).info
    for k, v in EXPECTED[name].items():
        assert info[k] == v, (k, info[k], v)
    assert info["mode"] == ("copy" if (w.alpha, w.beta) == (1.0, 0.0)
                            else "scale" if w.beta == 0 else "axpby")
    assert info["numel"] == w.numel
    if info["kernel"] == "tile" and w in WORKLOADS:  # the named workloads' runs start on lines
        assert info["vec_a"] == info["vec_b"] == 16 // w.elem_bytes
        assert info["lds_bytes"] <= 40 * 1024          # at least 4 workgroups per CU
        assert (info["run_b"] * w.elem_bytes) % 128 == 0   # B runs of whole lines
        assert (info["rows_per_pass"] * w.elem_bytes) % 128 == 0  # passes of whole lines
        # non-temporal A loads exactly when A runs are whole lines
        assert bool(info["hints"] & 2) == ((info["run_a"] * w.elem_bytes) % 128 == 0)
        assert info["hints"] & 1                        # non-temporal B stores
        assert info["lds_pitch"] % 2 == 1


def test_alpha_beta_rounded_to_dtype():
    p = hptt.create_plan((1, 0), (4, 4), alpha=0.1, beta=0.0, dtype="f32")
    assert p.info["mode"] == "scale"
    # 1 + 2^-30 rounds to 1.0 in float: a copy
    assert hptt.create_plan((1, 0), (4, 4), alpha=1 + 2 ** -30, dtype="f32").info["mode"] == "copy"
    assert hptt.create_plan((1, 0), (4, 4), alpha=1 + 2 ** -30, dtype="f64").info["mode"] == "scale"


def _raw_create(perm, size, dtype=0, options=None, n=None):
    lib = hptt.library()
    n = len(perm) if n is None else n
    pm = (ctypes.c_int32 * max(len(perm), 1))(*perm)
    sz = (ctypes.c_int64 * max(len(size), 1))(*size)
    h = ctypes.c_void_p(12345)
    if options is None:
        st = lib.hptt_create_plan(ctypes.byref(h), pm, n, sz, 1.0, 0.0, dtype)
    else:
        st = lib.hptt_create_plan_ex(ctypes.byref(h), pm, n, sz, 1.0, 0.0, dtype,
                                     ctypes.byref(options))
    return st, h


@pytest.mark.parametrize("perm,size,dtype,n", [
    ((0, 0), (2, 3), 0, None),       # not a permutation
    ((0, 2), (2, 3), 0, None),       # index out of range
    ((1, 0), (2, -1), 0, None),      # negative extent
    ((1, 0), (2, 3), 7, None),       # unknown dtype
    ((0,), (2,), 0, 0),              # N = 0
    (tuple(range(17)), (1,) * 17, 0, None),  # N above 16
])
def test_invalid_problems(perm, size, dtype, n):
    st, h = _raw_create(perm, size, dtype, n=n)
    assert st == 1 and not h.value


def test_null_arguments():
    lib = hptt.library()
    pm = (ctypes.c_int32 * 2)(1, 0)
    sz = (ctypes.c_int64 * 2)(2, 3)
    assert lib.hptt_create_plan(None, pm, 2, sz, 1.0, 0.0, 0) == 1
    h = ctypes.c_void_p()
    assert lib.hptt_create_plan(ctypes.byref(h), None, 2, sz, 1.0, 0.0, 0) == 1
    assert lib.hptt_create_plan(ctypes.byref(h), pm, 2, None, 1.0, 0.0, 0) == 1
    assert lib.hptt_plan_info(None, None) == 1
    assert lib.hptt_describe_plan(None, None, 0) == 1
    assert lib.hptt_destroy_plan(None) == 0


@pytest.mark.parametrize("field,value", [("kernel", 9), ("kernel", 1), ("run_a", -1),
                                         ("store_hint", 3), ("load_hint", -1), ("lds_pad", 65),
                                         ("max_blocks", -2), ("tile_order", 5), ("exact_runs", 2),
                                         ("row_passes", -1), ("row_passes", 65), ("block", 512),
                                         ("block", -1), ("skew", -1), ("skew", 1025),
                                         ("shear", 3), ("shear", -1), ("shared_runs", 3),
                                         ("shared_runs", -1)])
def test_invalid_options(field, value):
    opt = hptt.Options()
    setattr(opt, field, value)
    st, h = _raw_create((1, 0), (4, 4), options=opt)
    assert st == 1 and not h.value


def test_forced_kernel_that_does_not_apply():
    with pytest.raises(hptt.HpttError) as e:
        hptt.create_plan((0, 2, 1), (64, 5, 7), kernel="tile", shared_runs=2)
    assert e.value.status == 2
    # a kept stride-1 index is a shared index of a tile
    assert hptt.create_plan((0, 2, 1), (64, 5, 7), kernel="tile").info["shared_runs"] >= 1
    with pytest.raises(hptt.HpttError):
        hptt.create_plan((1, 0), (64, 5), kernel="stream")
    with pytest.raises(hptt.HpttError):
        hptt.create_plan((1, 0), (64, 5), kernel="axpby")
    assert hptt.create_plan((1, 0), (64, 5), kernel="generic").info["kernel"] == "generic"
    assert hptt.create_plan((0, 2, 1), (2, 5, 7), kernel="stream").info["kernel"] == "stream"


def test_exec_argument_checks_before_launch():
    """hptt_exec rejects bad arguments before touching the GPU."""
    lib = hptt.library()
    vp = ctypes.c_void_p
    assert lib.hptt_exec(None, vp(4096), vp(8192), None) == 1
    empty = hptt.create_plan((1, 0), (0, 5))
    assert lib.hptt_exec(empty.handle, None, None, None) == 0       # nothing to do
    p = hptt.create_plan((1, 0), (4, 4))
    assert lib.hptt_exec(p.handle, None, vp(1 << 20), None) == 1     # null A
    assert lib.hptt_exec(p.handle, vp(1 << 20), None, None) == 1     # null B
    assert lib.hptt_exec(p.handle, vp((1 << 20) + 2), vp(1 << 21), None) == 1   # misaligned
    assert lib.hptt_exec(p.handle, vp(1 << 20), vp((1 << 20) + 60), None) == 3  # overlap
    assert lib.hptt_exec(p.handle, vp(1 << 20), vp(1 << 20), None) == 3          # in place


def test_describe():
    d = hptt.create_plan((1, 0), (8192, 8192)).describe()
    assert "kernel=tile" in d and "fused=(8192,8192)" in d


def test_workload_bytes_follow_eq2():
    """Eq. (2): lambda = 2 when beta = 0 and 3 otherwise."""
    table = {float(b): int(l) for b, l in golden("eq2_lambda.txt")}
    for w in WORKLOADS:
        assert w.lam == table.get(w.beta, 3 if w.beta else 2)
        assert w.moved_bytes == w.lam * w.numel * w.elem_bytes


def test_plan_creation_is_quick():
    """The quick path of Section 3.1 keeps plan creation negligible: well
    under a millisecond even for large extents and rank 16."""
    import time
    cases = [((1 << 20, 1 << 12), (1, 0)), ((3, 5, 7, 11, 13, 17), (5, 4, 3, 2, 1, 0)),
             ((2,) * 16, tuple(range(15, -1, -1))), ((8192, 8192), (1, 0))]
    hptt.create_plan((1, 0), (4, 4))
    for size, perm in cases:
        t0 = time.perf_counter()
        for _ in range(10):
            hptt.create_plan(perm, size)
        assert (time.perf_counter() - t0) / 10 < 2e-3, size


# --------------------------------------------------------------------------
# Sub-tensors with outer sizes (Section 3.1, Fig. 3)
# --------------------------------------------------------------------------

def test_fig3b_outer_plan():
    rows = {r[0]: r[1:] for r in golden("fig3b_input.txt")}
    perm = tuple(int(x) for x in rows["perm"])
    size_a = tuple(int(x) for x in rows["sizeA"])
    outer_a = tuple(int(x) for x in rows["outerSizeA"])
    outer_b = tuple(int(x) for x in rows["outerSizeB"])
    info = hptt.create_plan(perm, size_a, outer_size_a=outer_a, outer_size_b=outer_b).info
    # A's sub-tensor spans from (0,0,0) to (7,15,15) of the 16x32x32 tensor
    assert info["footprint_a"] == 1 + 7 * 1 + 15 * 16 + 15 * 16 * 32
    assert info["footprint_b"] == 16 * 16 * 8
    assert info["ndim"] == 3 and info["kernel"] == "tile"


@pytest.mark.parametrize("outer_a,outer_b,fsize,fperm", [
    ((4, 5, 6), (5, 6, 4), (4, 30), (1, 0)),        # compact: A1, A2 fuse
    ((4, 8, 6), (5, 6, 4), (4, 5, 6), (1, 2, 0)),   # A1 padded in A: no fusion
    ((4, 5, 6), (7, 6, 4), (4, 5, 6), (1, 2, 0)),   # B's first index padded: no fusion
    ((4, 5, 6), (5, 6, 9), (4, 30), (1, 0)),        # padding only on B's last index
    ((9, 5, 6), (5, 6, 4), (4, 30), (1, 0)),        # padding on A0 does not stop A1+A2
])
def test_outer_fusion(outer_a, outer_b, fsize, fperm):
    info = hptt.create_plan((1, 2, 0), (4, 5, 6), outer_size_a=outer_a, outer_size_b=outer_b).info
    assert info["size"] == fsize and info["perm"] == fperm


def test_outer_smaller_than_size_rejected():
    with pytest.raises(hptt.HpttError):
        hptt.create_plan((1, 0), (4, 5), outer_size_a=(3, 5))
    with pytest.raises(hptt.HpttError):
        hptt.create_plan((1, 0), (4, 5), outer_size_b=(5, 3))


def test_strided_single_index_uses_generic():
    """A sub-tensor whose first extent is 1 leaves a strided index after the
    extent-1 index is dropped; the flat kernel must not serve it."""
    info = hptt.create_plan((0, 1), (1, 7), outer_size_a=(3, 7)).info
    assert info["kernel"] == "generic" and info["footprint_a"] == 1 + 6 * 3


def test_shear_only_where_b_runs_cannot_be_lines():
    """B runs are sheared onto lines only where they cannot be whole lines
    otherwise; never on the named workloads; never with shear = 2."""
    for w in WORKLOADS:
        assert hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype).info["shear"] == 0
    p = hptt.create_plan((1, 0), (39792, 1257), 1.0, 0.0, "f32")
    assert p.info["shear"] == 31 and p.info["run_b"] % 32 == 0
    assert p.info["hints"] & 1  # whole lines: non-temporal stores again
    p64 = hptt.create_plan((1, 0), (39792, 1257), 1.0, 0.0, "f64")
    assert p64.info["shear"] == 15
    assert hptt.create_plan((1, 0), (39792, 1257), 1.0, 0.0, "f32", shear=2).info["shear"] == 0
    assert hptt.create_plan((1, 0), (39792, 1280), 1.0, 0.0, "f32").info["shear"] == 0


def test_shared_runs_where_disjoint_runs_collapse():
    """Runs that share indices replace disjoint ones whose B run is shorter
    than a line (B's stride-1 extent 2 with its next index in the A run), or
    whose vectors are narrower, and the generic kernel on kept stride-1
    indices under 64 bytes; never on the named workloads, never with
    shared_runs = 2."""
    for w in WORKLOADS:
        assert hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype).info["shared_runs"] == 0
    # 12x3x2x2293x303, perm [2,1,4,3,0]: disjoint runs write 8-byte B runs
    size, perm = (12, 3, 2, 2293, 303), (2, 1, 4, 3, 0)
    d = hptt.create_plan(perm, size, 1.0, 1.0, "f32", shared_runs=2).info
    assert d["run_b"] * 4 < 128 and d["shared_runs"] == 0
    s = hptt.create_plan(perm, size, 1.0, 1.0, "f32").info
    assert s["kernel"] == "tile" and s["shared_runs"] == 2
    assert s["run_a"] * 4 >= 512 and s["run_b"] * 4 >= 512 and s["lds_bytes"] <= 20 * 1024
    # beta = 0 takes the larger budget
    assert hptt.create_plan(perm, size, 1.0, 0.0, "f32").info["lds_bytes"] <= 40 * 1024
    # a kept stride-1 index of 8 bytes
    k = hptt.create_plan((0, 2, 1), (2, 60251, 415), 1.0, 1.0, "f32").info
    assert k["kernel"] == "tile" and k["shared_runs"] == 1
    # 2-element A runs read one element per lane; shared runs take 16 bytes
    n = hptt.create_plan((1, 0, 2), (2, 44, 570480), 1.0, 1.0, "f32").info
    assert n["shared_runs"] == 3 and n["vec_a"] == 4 and n["vec_b"] == 4
    # short A runs whose rows follow each other in A stay disjoint
    assert hptt.create_plan((1, 0), (14, 3582084), 1.0, 1.0, "f32").info["shared_runs"] == 0
    assert hptt.create_plan(perm, size, 1.0, 1.0, "f32", shared_runs=2).info["shared_runs"] == 0


def test_flat_stream_walk_rule():
    """Kernel S walks B flat where the kept rows would move one element per
    access (odd rows), or two fp32 elements; not for rows that take whole
    vectors, not where B is a sub-tensor with gaps, and not when switched
    off."""
    odd = hptt.create_plan((0, 3, 2, 1), (75, 100, 11, 60), 1.0, 0.0, "f32")
    assert odd.info["kernel"] == "stream" and odd.info["flat_runs"] == 1
    assert odd.info["vec_b"] == 4 and odd.info["tiles"] == -(-odd.numel // 4)
    assert "flat=1" in odd.describe()
    assert hptt.create_plan((0, 3, 2, 1), (75, 100, 11, 60), 1.0, 0.0, "f32",
                            flat_runs=2).info["flat_runs"] == 0
    assert hptt.create_plan((0, 3, 2, 1), (95, 96, 9, 9), 2.0, 0.5, "f64").info["flat_runs"] == 1
    assert hptt.create_plan((0, 3, 2, 1), (96, 96, 9, 9), 2.0, 0.5, "f64").info["flat_runs"] == 0
    assert hptt.create_plan((0, 3, 2, 1), (96, 96, 9, 9), 1.0, 0.0, "f32").info["flat_runs"] == 0
    # two fp32 elements per access: flat in both update modes; two fp64
    # elements (whole vectors) keep the row walk
    assert hptt.create_plan((0, 3, 2, 1), (66, 10, 9, 9), 1.0, 0.0, "f32").info["flat_runs"] == 1
    assert hptt.create_plan((0, 3, 2, 1), (66, 10, 9, 9), 1.0, 1.0, "f32").info["flat_runs"] == 1
    assert hptt.create_plan((0, 3, 2, 1), (66, 10, 9, 9), 1.0, 0.0, "f64").info["flat_runs"] == 0
    forced = hptt.create_plan((0, 3, 2, 1), (96, 96, 9, 9), 1.0, 0.0, "f32", flat_runs=1)
    assert forced.info["flat_runs"] == 1
    gaps = hptt.create_plan((0, 2, 1), (63, 5, 7), 1.0, 0.0, "f32", outer_size_b=(64, 7, 5))
    assert gaps.info["kernel"] == "stream" and gaps.info["flat_runs"] == 0


def test_flat_b_runs_rule():
    """Flat B runs where the inner B extents are not whole lines (the 6-D
    workload), not where they are, not when switched off, and never when the
    flattened range exceeds 32-bit positions."""
    p = hptt.create_plan((5, 2, 0, 4, 1, 3), (24, 20, 16, 24, 18, 20), 1.5, 0.0, "f32")
    assert p.info["flat_runs"] == 2 and p.info["run_b"] == 32
    assert "flat=2" in p.describe()
    off = hptt.create_plan((5, 2, 0, 4, 1, 3), (24, 20, 16, 24, 18, 20), 1.5, 0.0, "f32",
                           flat_runs=2)
    assert off.info["flat_runs"] == 0 and off.info["run_b"] == 160
    # inner B extent of 32 fp32 = one line: the usual runs already are lines
    whole = hptt.create_plan((5, 2, 0, 4, 1, 3), (24, 20, 16, 24, 18, 32), 1.5, 0.0, "f32")
    assert whole.info["flat_runs"] == 0
    # 20 x 300,000,000 flattened positions: beyond 32 bits, no flat runs even when asked
    big = hptt.create_plan((1, 3, 0, 2), (24, 20, 7, 300_000_000), 1.0, 0.0, "f32",
                           flat_runs=1)
    assert big.info["flat_runs"] == 0
    small = hptt.create_plan((1, 3, 0, 2), (24, 20, 7, 3000), 1.0, 0.0, "f32", flat_runs=1)
    assert small.info["flat_runs"] == 2


@pytest.mark.parametrize("size_a,perm,dtype,whole", [
    ((66, 757576), (1, 0), "f32", 66),       # one-line target would cut 66 into 33 + 33
    ((69, 988, 733), (1, 2, 0), "f32", 69),
    ((30, 2762, 85, 7), (1, 2, 3, 0), "f64", 30),
])
def test_sheared_tiles_keep_a_short_stride1_index_whole(size_a, perm, dtype, whole):
    """Sheared tiles take a stride-1 A index that the one-line A-run target
    would cut in two whole, with B runs of two lines (the next A index is the
    B run's, so a tile's A rows are one contiguous block); an index cut in
    three keeps the cut."""
    for beta in (0.0, 1.0):
        i = hptt.create_plan(perm, size_a, 1.0, beta, dtype).info
        assert i["shear"] > 0 and i["run_a"] == whole, i
        assert i["run_b"] >= 128 // i["elem_bytes"] * 2
    # a B-run target given by the caller is kept
    assert hptt.create_plan(perm, size_a, 1.0, 0.0, dtype, run_b=256).info["run_b"] > 64
    i = hptt.create_plan((1, 0), (87, 30000), 1.0, 0.0, "f32").info
    assert i["shear"] > 0 and i["run_a"] == 29


def test_shared_runs_budget_with_b_read():
    """fp32 shared-run tiles of one or two rows take 40 KiB of LDS when B is
    read (the usual budget then is 20 KiB); taller tiles and fp64 do not."""
    one = hptt.create_plan((1, 3, 0, 2), (2, 26250, 4, 238), 1.0, 1.0, "f32").info
    assert one["shared_runs"] and one["rows_per_pass"] == 1 and one["lds_bytes"] > 20 * 1024
    assert hptt.create_plan((1, 3, 0, 2), (2, 26250, 4, 238), 1.0, 0.0,
                            "f32").info["lds_bytes"] <= 40 * 1024
    tall = hptt.create_plan((2, 1, 4, 3, 0), (12, 3, 2, 2293, 303), 1.0, 1.0, "f32").info
    assert tall["shared_runs"] and tall["rows_per_pass"] > 2 and tall["lds_bytes"] <= 20 * 1024
    f64 = hptt.create_plan((3, 0, 1, 4, 2), (10, 71, 2, 2, 17606), 1.0, 1.0, "f64").info
    assert f64["shared_runs"] and f64["rows_per_pass"] <= 2 and f64["lds_bytes"] <= 20 * 1024


@pytest.mark.parametrize("size_a,perm,want", [
    # the window of resident tiles touches far fewer B regions with A4 first
    ((24, 20, 16, 24, 18, 20), (5, 2, 0, 4, 1, 3), 2),
    # B order: A0 (outer, B-adjacent) before A2
    ((427, 110, 3, 355), (3, 2, 1, 0), 3),
    # 10-element A runs: A order keeps A3 (A-adjacent) first
    ((2, 5, 9, 15, 220, 168), (2, 4, 1, 0, 5, 3), 1),
    ((6, 5126, 2, 3, 7, 39), (5, 1, 2, 4, 0, 3), 1),
    ((8192, 8192), (1, 0), 1),
])
def test_grid_order_choice(size_a, perm, want):
    """The quick path orders the outer grid digits by the regions of A and B
    a window of resident tiles touches (A order unless another order has at
    most 0.8 times as many); forced orders are kept."""
    assert hptt.create_plan(perm, size_a).info["grid_order"] == want
    for forced in (1, 2, 3):
        assert hptt.create_plan(perm, size_a, grid_order=forced).info["grid_order"] == forced
    with pytest.raises(hptt.HpttError):
        hptt.create_plan(perm, size_a, grid_order=4)


def test_hptt_log_prints_each_plan():
    """HPTT_LOG=1 prints every new plan (fused shape, kernel, tile, grid) to
    stderr; unset or "0" prints nothing."""
    import subprocess
    import sys
    code = ("from paper_1704_04374_amd import hptt; "
            "hptt.create_plan((1, 0), (64, 32)); hptt.create_plan((2, 0, 1), (48, 40, 32))")
    for val, lines in (("1", 2), ("0", 0), (None, 0)):
        env = {k: v for k, v in os.environ.items() if k != "HPTT_LOG"}
        if val is not None:
            env["HPTT_LOG"] = val
        r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True,
                           text=True, timeout=120)
        assert r.returncode == 0, r.stderr
        got = [ln for ln in r.stderr.splitlines() if ln.startswith("[hptt] plan: ")]
        assert len(got) == lines, r.stderr
        if lines:
            assert "fused=(64,32) perm=(1,0)" in got[0] and "kernel=tile" in got[0]
            assert "fused=(1920,32) perm=(1,0)" in got[1]


def test_xcd_group_rule():
    """Tiles whose A runs are at most 320 bytes and do not start on 128-byte
    lines are dealt to the XCDs 16 at a time in grid-digit order; aligned
    runs, longer runs and shared-run tiles keep the diagonal round robin;
    forced values are kept, and the contiguous XCD ranges of tile orders 3
    and 4 replace the groups."""
    for beta in (0.0, 1.0):
        short = hptt.create_plan((1, 0), (2193, 22800), 1.0, beta).info
        assert short["xcd_group"] == 16 and short["tile_order"] == 1, short
        assert short["run_a"] * 4 <= 256
        mid = hptt.create_plan((1, 0), (66, 757576), 1.0, beta).info    # 264-byte runs
        assert mid["xcd_group"] == 16 and 256 < mid["run_a"] * 4 <= 320, mid
        f64 = hptt.create_plan((3, 1, 0, 2), (77, 1651, 2, 99), 1.0, beta, "f64").info
        assert f64["xcd_group"] == 16 and f64["run_a"] * 8 <= 320, f64
    assert hptt.create_plan((1, 0), (8192, 8192)).info["xcd_group"] == 1       # whole lines
    long_run = hptt.create_plan((3, 2, 1, 4, 0, 5), (6, 55, 48, 6, 7, 75)).info  # 672 bytes
    assert long_run["run_a"] * 4 > 320 and long_run["xcd_group"] == 1, long_run
    assert long_run["tile_order"] == 2
    # columns a multiple of 4 KiB apart in B (64 KiB here) keep the diagonal
    for beta in (0.0, 1.0):
        pow2 = hptt.create_plan((1, 0), (3001, 16384), 1.0, beta).info
        assert pow2["xcd_group"] == 1 and pow2["tile_order"] == 2, pow2
    assert hptt.create_plan((1, 0), (3001, 16384), 1.0, 1.0).info["run_a"] * 4 <= 320
    shared = hptt.create_plan((1, 3, 0, 2), (2, 26250, 4, 238)).info        # long runs
    assert shared["shared_runs"] and shared["xcd_group"] == 1
    for beta in (0.0, 1.0):  # kept-index shared-run tiles with 256-byte runs off the lines
        kept = hptt.create_plan((0, 2, 1), (2, 60251, 415), 1.0, beta).info
        assert kept["shared_runs"] and kept["run_a"] * 4 <= 320 and kept["xcd_group"] == 16, kept
    forced = hptt.create_plan((1, 0), (2193, 22800), xcd_group=1).info
    assert forced["xcd_group"] == 1 and forced["tile_order"] == 2
    forced = hptt.create_plan((1, 0), (8192, 8192), xcd_group=64).info
    assert forced["xcd_group"] == 64 and forced["tile_order"] == 2
    ranges = hptt.create_plan((1, 0), (2193, 22800), tile_order=3, xcd_group=16).info
    assert ranges["xcd_group"] == 0 and ranges["tile_order"] == 3
    for bad in (3, 12, 2048, -1):
        with pytest.raises(hptt.HpttError):
            hptt.create_plan((1, 0), (64, 32), xcd_group=bad)


def test_stream_xcd_groups_are_an_option():
    """Kernel S deals its blocks to the XCDs in groups only when asked (the
    quick path keeps plain round robin), and the autotuner lists the groups
    and the flat and row walks as distinct candidates."""
    perm, size = (0, 4, 3, 1, 2), (42, 4, 13, 1067, 21)
    assert hptt.create_plan(perm, size).info["xcd_group"] == 1
    p = hptt.create_plan(perm, size, xcd_group=64).info
    assert p["kernel"] == "stream" and p["xcd_group"] == 64
    cands = hptt.autotune_candidates(perm, size, 1.0, 0.0, "f32")
    got = [c for c in cands if c.get("xcd_group") in (16, 64)]
    assert len(got) == 2, cands
    assert any(c.get("flat_runs") == 2 for c in cands), cands
