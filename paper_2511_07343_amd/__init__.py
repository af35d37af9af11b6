"""TNT hierarchical memory layer on MI355X: HIP kernels behind a C ABI
(``include/tnt.h``) and a thin ctypes binding (``tnt.py``).

Importing the package loads nothing; ``paper_2511_07343_amd.tnt.lib()`` loads
the built ``libtnt.so`` and raises if it is missing.
"""
__all__ = ["inputs", "tnt", "build"]
