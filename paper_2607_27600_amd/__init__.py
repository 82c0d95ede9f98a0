"""MI355X (gfx950) implementation of the counter-causal refresh-scoring pass.

The work is done by the HIP kernels of libcc.so behind the C ABI in include/cc.h;
:mod:`paper_2607_27600_amd.cc` is its ctypes binding.
"""
