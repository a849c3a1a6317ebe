"""MI355X-native Speculative Probing classification forward.

The compute lives in ``libsp_probe.so`` (HIP kernels for gfx950 behind a C ABI,
``include/sp_probe.h``); ``paper_2608_28099_amd.binding`` is the thin ctypes
layer over it.  ``configs`` and ``inputs`` describe and generate workloads.
Importing this package loads nothing; the binding loads the library on first use
and raises if it is missing.
"""
