"""DBLast head + stochastic verification on AMD MI355X (gfx950).

The computation lives in libdblast.so (HIP kernels behind the C ABI of include/dblast.h);
``paper_2608_05448_amd.dblast`` is its Python binding and ``paper_2608_05448_amd.build``
compiles it. Importing this package loads nothing; the first call through the binding loads
the library and fails loudly if it is missing.
"""
