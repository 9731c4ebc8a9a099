"""MI355X (gfx950) fused store-path library: expert-parallel dispatch / grouped GEMM /
combine, GEMM scatter epilogues and store pacing, as a C-ABI shared library
(libxstage.so, include/xstage.h) with a thin ctypes binding (``xstage``) and a
buffer-owning helper for the EP layer (``layer``)."""
