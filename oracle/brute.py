"""Pure-Python brute force of Eq. (1) of the HPTT paper, for tiny tensors.

TEST INFRASTRUCTURE, NOT PRODUCT CODE: a second, independent spelling of the
definition, used to cross-check the C oracle on every permutation of small
rank.  It walks every A multi-index with ``itertools.product``, places the
element at the B multi-index whose k-th entry is A's index ``perm[k]``
(Table 1: position k of B carries A index perm[k]) and applies
``alpha*a + beta*b`` with numpy scalars of the tensor dtype, so each product
and the sum are rounded once in that precision (no fused multiply-add).
Offsets follow the Fortran layout of Section 1.
"""
from __future__ import annotations

import itertools

import numpy as np


def _offset(index, sizes):
    off, stride = 0, 1
    for i, n in zip(index, sizes):
        off += i * stride
        stride *= n
    return off


def transpose(A, size_a, perm, alpha=1.0, beta=0.0, B=None, dtype=np.float32):
    """Return B (a flat list of numpy scalars of ``dtype``) after Eq. (1)."""
    size_b = [size_a[p] for p in perm]
    numel = 1
    for n in size_a:
        numel *= n
    al, be = dtype(alpha), dtype(beta)
    out = [dtype(0)] * numel if B is None else [dtype(x) for x in B]
    # itertools.product varies the last entry fastest; reverse to get the
    # Fortran order (first index fastest).  The order does not change the
    # result since each B element is written exactly once.
    for rev in itertools.product(*[range(n) for n in reversed(size_a)]):
        i = tuple(reversed(rev))
        j = tuple(i[p] for p in perm)
        a = dtype(A[_offset(i, size_a)])
        ob = _offset(j, size_b)
        if be == 0:
            out[ob] = a if al == 1 else dtype(al * a)
        else:
            out[ob] = dtype(dtype(al * a) + dtype(be * out[ob]))
    return out
