"""MI355X (gfx950) implementation of the SonicMoE layer (arXiv 2512.14080).

The layer -- token-choice top-K router, token rounding, gather-fused grouped
GEMMs with SwiGLU / dSwiGLU / dS epilogues and gather-and-sum aggregation,
forward and backward -- runs in hand-written HIP kernels behind the C ABI of
include/sonicmoe.h (libsonicmoe.so).  ``binding`` is the ctypes binding,
``layer`` allocates one layer's device buffers, ``workloads`` holds the
seeded synthetic inputs and ``build`` compiles the library.
"""
