"""MI355X (gfx950) CCI-sparse forward path: packing, CCI-sparse product and
implicit-im2col convolution as hand-written HIP kernels behind a C ABI
(include/cci.h).  ``paper_1910_11971_amd.cci`` is the Python binding; importing
it loads ``libcci.so`` and fails loudly if it has not been built."""

__all__ = ["cci", "workloads"]
