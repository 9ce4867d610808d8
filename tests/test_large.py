"""Problems beyond 2^31 and 2^32 elements, on the CPU: the kernels' index
arithmetic (emulated by the host emulator, offsets only) for plans whose
numbers no longer fit 32 bits.  Eq. (1) puts no bound on the extents; the
plan builder keeps every 32-bit quantity a kernel uses (in-tile offsets, tile
and item counts, digit extents) below its limit or takes a 64-bit variant.

  - a 2-D transposition just above 2^31 elements: every workgroup run, every
    B element written exactly once (the tile kernel's 64-bit offset variant);
  - above 2^32 elements: a 2-D transposition, a 3-D one with a short fused
    A run, a stride-1-kept problem and an identity (axpby) problem, each on a
    stride of workgroups and on the last one, every access in bounds and
    aligned."""
from __future__ import annotations

import numpy as np
import pytest

from emulator import emu




def test_tile_just_above_2_31_elements_covers_b_once():
    size, perm = (46341, 46341), (1, 0)          # 2,147,488,281 elements
    assert size[0] * size[1] > 2 ** 31
    p = emu.plan(perm, size, 1.0, 0.0, "f32")
    assert p.info["kernel"] == "tile"
    err, msg, cnt = emu.run(p, counts=True)
    assert err == 0, msg
    assert cnt.min() == 1 and cnt.max() == 1


@pytest.mark.parametrize("size,perm,dtype,kernel", [
    ((65537, 65537), (1, 0), "f32", "tile"),
    ((3, 65537, 21846), (0, 2, 1), "f32", "tile"),
    ((2, 2147483649), (1, 0), "f32", "tile"),
    ((64, 1024, 256, 257), (0, 2, 1, 3), "f32", "stream"),
    ((4294971392,), (0,), "f32", "axpby"),
    ((32768, 65537, 2), (1, 0, 2), "f64", None),
], ids=lambda x: "x".join(map(str, x)) if isinstance(x, tuple) else str(x))
@pytest.mark.parametrize("beta", [0.0, 1.0])
def test_above_2_32_elements_in_bounds(size, perm, dtype, kernel, beta):
    n = int(np.prod(size))
    assert n > 2 ** 32
    p = emu.plan(perm, size, 1.0, beta, dtype)
    if kernel:
        assert p.info["kernel"] == kernel
    grid = p.info["grid"]
    # about 1500 workgroups from the first on, then the first and the last
    for stride in (max(1, grid // 1500), max(1, grid - 1)):
        err, msg, _ = emu.run(p, block_stride=stride)
        assert err == 0, f"{p.describe()} (workgroup stride {stride}): {msg}"


@pytest.mark.parametrize("va", [1, 2])
def test_stream_slabs_beyond_2_32_items(va):
    """The stride-1-kept walk at a width whose items exceed 32 bits (here the
    widths a misaligned pointer narrows to) launches once per slab of the
    slowest B positions: a 64 x 4096 x 16385 fp32 problem (2^32 + 2^18
    elements) at 1-element vectors covered whole, every B element written
    exactly once; at 2-element vectors on a stride of workgroups."""
    size, perm = (64, 4096, 16385), (0, 2, 1)
    p = emu.plan(perm, size, 1.0, 0.0, "f32")
    assert p.info["kernel"] == "stream" and p.info["vec_a"] == 4
    if va == 1:
        err, msg, cnt = emu.run(p, va=1, vb=1, counts=True, mis_a=1, mis_b=1)
        assert err == 0, msg
        assert cnt.min() == 1 and cnt.max() == 1
    else:
        for stride in (997, max(1, p.info["grid"] - 1)):
            err, msg, _ = emu.run(p, va=2, vb=2, block_stride=stride, mis_a=2, mis_b=2)
            assert err == 0, msg
