"""Fused fp16 GEMM + bias + ReLU for AMD MI355X (gfx950).

The compute lives in the HIP library ``libgba.so`` (C ABI declared in
``include/gba.h``); :mod:`paper_2006_12645_amd.gba` is a thin ctypes binding
over it.
"""
