"""SCOPE sparse self-attention for video DiTs on MI355X (gfx950).

The layer runs in hand-written HIP kernels behind the C ABI of
include/scope.h (libscope.so, built by ``build.py``).  ``binding`` is the
ctypes binding of that ABI, ``layer`` sequences its five calls, and
``inputs`` generates seeded synthetic workloads.
"""
