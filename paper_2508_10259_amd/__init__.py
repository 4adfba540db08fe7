"""Cached-context action decoder for one AMD MI355X (gfx950).

The decoder's every arithmetic step runs in ``libams.so`` (hand-written HIP
kernels behind the C ABI in ``include/ams.h``).  ``capi`` is the ctypes
binding, ``runtime`` the torch-facing wrapper (device memory and streams
only), ``workload`` the seeded synthetic inputs and ``build`` the hipcc
build.  Importing the package loads nothing; ``capi.load()`` does, and fails
loudly when the library is missing.
"""
