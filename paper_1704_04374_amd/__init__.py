"""MI355X (gfx950) tensor transposition, Eq. (1) of the HPTT paper:
B_{Pi(i_1..i_N)} <- alpha*A_{i_1..i_N} + beta*B_{Pi(i_1..i_N)}, Fortran layout.

The work runs in hand-written HIP kernels behind the C ABI of include/hptt.h;
``paper_1704_04374_amd.hptt`` is its Python binding.
"""
from .hptt import HpttError, Plan, create_plan, transpose  # noqa: F401
