"""MI355X (gfx950) implementation of FoX attention with adaptive computation pruning.

The compute lives in the HIP library ``libacp.so`` built from ``csrc/``; the
Python module ``acp`` is a thin ctypes binding with the C ABI's names.  Nothing
is loaded at import time: the library is opened on first use, and every entry
point raises if it is missing.
"""
__all__ = ["acp", "workloads"]
