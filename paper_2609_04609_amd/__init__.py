"""CIERA exponent-reuse codec for bf16 weight shards on MI355X (gfx950).

The codec itself lives in ``libciera.so`` (hand-written HIP kernels behind a
C ABI, declared in ``include/ciera.h``); ``ciera`` is its ctypes binding and
``synth`` the seeded input generators. Importing the package loads nothing:
the library is opened on first use and a missing build raises.
"""
