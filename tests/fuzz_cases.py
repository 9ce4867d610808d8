"""Seeded random transposition problems for the fuzz tests: rank 1-7,
extents around vector and line sizes, random permutations, fp32 and fp64,
every update mode, random plan options, sub-tensors of padded enclosing
tensors, and base pointers 0-3 elements off a 256-byte boundary.  Problem
descriptions only: no part of the transposition is computed here."""
from __future__ import annotations

import math

import numpy as np

EXTENTS = [1, 2, 3, 4, 5, 7, 8, 9, 15, 16, 17, 31, 32, 33, 48, 63, 64, 65, 96, 127, 128, 129,
           255, 256, 300, 1000, 1024, 4099]
MAX_NUMEL = 1 << 21
UPDATES = [(1.0, 0.0), (1.5, 0.0), (1.0, 1.0), (-0.75, 1.25), (2.0, 0.5), (0.0, 1.0)]


def case(seed: int, i: int) -> dict:
    """Case i of the set `seed` (odd seeds allow extent-1 indices and the
    identity permutation freely; even seeds mostly real transpositions)."""
    rng = np.random.default_rng([seed, i])
    ext = EXTENTS if seed % 2 else [e for e in EXTENTS if e > 1] + [1]
    while True:
        n = int(rng.integers(1 if seed % 2 else 2, 8))
        size = [int(rng.choice(ext)) for _ in range(n)]
        if 0 < math.prod(size) <= MAX_NUMEL:
            break
    while True:
        perm = [int(p) for p in rng.permutation(n)]
        if seed % 2 or n == 1 or perm != list(range(n)):
            break
    dtype = "f32" if rng.random() < 0.6 else "f64"
    alpha, beta = UPDATES[int(rng.integers(0, len(UPDATES)))]
    knobs = {}
    if rng.random() >= 0.45:
        for k in rng.choice(["run", "shear", "flat", "shared", "gorder", "order", "block", "depth",
                             "hints", "vec", "kernel", "passes", "maxblocks", "xcd"],
                            size=int(rng.integers(1, 3)), replace=False):
            if k == "run":
                knobs["run_a"] = int(rng.choice([4, 8, 16, 32, 64, 128, 256]))
                knobs["run_b"] = int(rng.choice([4, 8, 16, 32, 64, 128]))
            elif k == "shear":
                knobs["shear"] = int(rng.choice([1, 2]))
            elif k == "flat":
                knobs["flat_runs"] = int(rng.choice([1, 2]))
            elif k == "shared":
                knobs["shared_runs"] = int(rng.choice([1, 2]))
            elif k == "gorder":
                knobs["grid_order"] = int(rng.integers(1, 4))
            elif k == "order":
                knobs["tile_order"] = int(rng.integers(1, 5))
            elif k == "block":
                knobs["block"] = 1024
            elif k == "depth":
                knobs["depth"] = int(rng.integers(2, 6))
            elif k == "hints":
                knobs["store_hint"] = int(rng.integers(1, 3))
                knobs["load_hint"] = int(rng.integers(1, 3))
            elif k == "vec":
                knobs["max_vec"] = int(rng.choice([1, 2]))
            elif k == "kernel":
                knobs["kernel"] = str(rng.choice(["generic", "tile", "stream"]))
            elif k == "passes":
                knobs["row_passes"] = int(rng.integers(2, 4))
            elif k == "maxblocks":
                knobs["max_blocks"] = int(rng.choice([1, 7, 64, 300]))
            elif k == "xcd":
                knobs["xcd_group"] = int(rng.choice([2, 16, 1024]))
    outer = None
    if rng.random() < 0.2:
        size_b = [size[p] for p in perm]
        oa = [s + int(rng.choice([0, 0, 1, 3, 8])) for s in size]
        ob = [s + int(rng.choice([0, 0, 1, 3, 8])) for s in size_b]
        sa = [int(rng.integers(0, o - s + 1)) for s, o in zip(size, oa)]
        sb = [int(rng.integers(0, o - s + 1)) for s, o in zip(size_b, ob)]
        if math.prod(oa) <= 2 * MAX_NUMEL and math.prod(ob) <= 2 * MAX_NUMEL:
            outer = (oa, ob, sa, sb)
    return dict(size=size, perm=perm, dtype=dtype, alpha=alpha, beta=beta, knobs=knobs,
                outer=outer, off_a=int(rng.integers(0, 4)), off_b=int(rng.integers(0, 4)))


def fortran_offset(index, extents) -> int:
    off, stride = 0, 1
    for i, e in zip(index, extents):
        off += int(i) * stride
        stride *= int(e)
    return off


def plan_kwargs(c: dict) -> dict:
    kw = dict(c["knobs"])
    if c["outer"]:
        kw["outer_size_a"], kw["outer_size_b"] = c["outer"][0], c["outer"][1]
    return kw


def first_elements(c: dict):
    """Element offsets of the sub-tensors' first elements from the starts of
    the buffers (pointer offset plus start inside the enclosing tensor), and
    the buffers' lengths in elements."""
    if c["outer"]:
        oa, ob, sa, sb = c["outer"]
        return (c["off_a"] + fortran_offset(sa, oa), c["off_b"] + fortran_offset(sb, ob),
                c["off_a"] + math.prod(oa), c["off_b"] + math.prod(ob))
    n = math.prod(c["size"])
    return c["off_a"], c["off_b"], c["off_a"] + n, c["off_b"] + n
