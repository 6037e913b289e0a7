"""CRISP sparse prefill attention for AMD MI355X (gfx950).

The compute path is libcrisp.so (HIP kernels behind the C ABI of
include/crisp.h); `paper_2609_01925_amd.crisp` is its Python binding.
"""
__all__ = ["crisp"]
