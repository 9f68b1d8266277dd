"""FP64 matrix multiplication emulated with Ozaki scheme II on the FP4 (E2M1)
matrix cores of the AMD Instinct MI355X (gfx950), through base-13 FP4 limbs.

The compute path is the HIP library ``libozfp4.so`` (C ABI declared in
``include/ozfp4.h``); ``paper_2608_06812_amd.ozfp4`` is its thin Python
binding. There is no CPU fallback: the binding raises if the library is
missing.
"""
