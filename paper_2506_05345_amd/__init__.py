"""Dynamic Memory Sparsification (DMS) decode / prefill on AMD MI355X (gfx950).

The compute path is libdms.so (HIP kernels behind a C ABI, ``include/dms.h``);
``paper_2506_05345_amd.dms`` is its Python binding.
"""
from . import dms  # noqa: F401
