"""DiffKV decode hot path for MI355X (gfx950).

The compute lives in the HIP library libdiffkv.so built from csrc/; the
Python module `diffkv` is a thin ctypes binding over its C ABI
(include/diffkv.h).  Importing the binding does not load the library; the
first call does, and raises if it is missing.
"""
