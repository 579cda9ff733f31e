"""MiKV mixed-precision KV-cache decode path for MI355X (gfx950).

The compute lives in ``libmikv.so`` (HIP kernels behind a C ABI, declared in
``include/mikv.h``).  ``paper_2402_18096_amd.mikv`` is the thin ctypes binding;
``paper_2402_18096_amd.workloads`` holds the seeded synthetic inputs.  Importing
this package loads nothing: the binding loads the library on first use and
raises if it has not been built.
"""
