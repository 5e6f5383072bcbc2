"""MI355X-native view-masked attention and fused token log-prob (MemoryWalker,
arXiv 2609.00865).  ``mv`` is the binding of libmv (HIP kernels for gfx950 and
the C ABI declared in include/mv.h); ``synth`` draws seeded synthetic inputs;
``build`` compiles libmv.so in-tree."""
