"""MI355X (gfx950) implementation of MOPAR's sliced inference hot path.

The computation runs in libmopar.so (hand-written HIP); this package is its
Python binding.  See include/mopar.h for the C ABI.
"""
from ._lib import MoparError, lib  # noqa: F401
from .binding import (SlicedModel, boundary_to_canonical, make_codec, make_plan,  # noqa: F401
                      mopar_boundary_code_bytes, mopar_boundary_decode, mopar_boundary_encode,
                      mopar_plan_slices, mopar_subslice_range, tensor_desc)
