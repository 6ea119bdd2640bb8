"""DP-SGD-RC randomized per-sample norm estimation on AMD MI355X (gfx950).

The compute lives in libdprc.so (hand-written HIP, C ABI in include/dprc.h);
``paper_2605_24879_amd.dprc`` is its Python binding.
"""

from . import dprc  # noqa: F401
