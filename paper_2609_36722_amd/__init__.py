"""Attuner suffix prefill over a frozen position-independent artifact cache,
for AMD Instinct MI355X (gfx950).

The compute path is libattuner.so (hand-written HIP kernels behind the C ABI
of include/attuner.h); :mod:`paper_2609_36722_amd.api` is its Python binding.
"""

from ._lib import LIB_PATH  # noqa: F401
