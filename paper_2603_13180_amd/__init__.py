"""MXNorm on MI355X (gfx950): fused RMS-estimate + MX cast kernels.

The compute lives in ``libmxnorm.so`` (hand-written HIP kernels behind a C
ABI declared in ``include/mxnorm.h``).  ``paper_2603_13180_amd.mxnorm`` is a
thin ctypes binding with the same entry-point names; it loads the library on
first use and raises if the library is missing or no GPU is present -- there
is no CPU fallback.  ``paper_2603_13180_amd.synth`` draws seeded synthetic
inputs.
"""
