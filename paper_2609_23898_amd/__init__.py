"""CERAR, the coded approximate ring all-reduce, on MI355X (gfx950).

``paper_2609_23898_amd.cerar``  ctypes binding of the in-tree libcerar.so
                                 (HIP kernels + C ABI declared in include/cerar.h)
``paper_2609_23898_amd.synth``   seeded synthetic gradients shaped like the
                                 paper's workloads
``paper_2609_23898_amd.build``   compiles libcerar.so with hipcc for gfx950
"""
