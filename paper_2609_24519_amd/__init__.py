"""Exact integer matrix products as a few FP4 (E2M1) GEMMs on MI355X (gfx950).

The HIP library ``libawe.so`` (kernels + C ABI, declared in ``include/awe.h``)
does all the work; ``awe`` is a thin ctypes binding with the same names.
Importing this package does not load the library; ``awe.lib()`` does, and it
raises if the library has not been built.
"""
