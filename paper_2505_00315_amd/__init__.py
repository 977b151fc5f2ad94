"""MI355X (gfx950) Mixture of Sparse Attention layer: HIP kernels behind a C ABI
(include/mosa.h) with a thin ctypes binding (``paper_2505_00315_amd.mosa``)."""
