"""libreqat: microscaled-FP4 (MXFP4 / NVFP4) quantize, fake-quant and W4A4 GEMM
for AMD Instinct MI355X (gfx950).

The compute lives in the HIP shared library ``libreqat.so`` (C ABI declared in
``include/reqat.h``); :mod:`paper_2606_15682_amd.reqat` is the thin ctypes
binding.  Importing this package loads nothing; the binding loads the library
on first use and raises if it has not been built.
"""
__all__ = ["reqat", "workloads"]
