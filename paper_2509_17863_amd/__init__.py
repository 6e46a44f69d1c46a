"""MI355X-native expert-server forward step (EaaS, arXiv 2509.17863).

The compute path is libeaas.so (HIP kernels for gfx950 behind the C ABI in
include/eaas.h); ``eaas`` is its Python binding and ``synth`` the seeded
synthetic input generator.
"""
