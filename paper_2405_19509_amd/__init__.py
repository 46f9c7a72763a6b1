"""Partial-straggler gradient coding on AMD MI355X (gfx950).

The hot path lives in the HIP library libgcx.so behind the C ABI of
include/gcx.h; ``paper_2405_19509_amd.gcx`` is its Python binding.
"""
from . import gcx  # noqa: F401  (the binding loads libgcx.so lazily, on first call)
