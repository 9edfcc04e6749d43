"""FastTPS token-phase decoder layer for MI355X (gfx950).

The compute path is ``libfasttps.so`` (HIP kernels behind a C ABI, declared in
``include/fasttps.h``); ``layer`` is a thin ctypes binding over it that only
marshals arguments. ``configs`` and ``inputs`` hold workload shapes and the
seeded synthetic input generator. Importing this package does not load the
library; ``layer`` does, and raises if it is missing.
"""
__all__ = ["configs", "inputs"]
