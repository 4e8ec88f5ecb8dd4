"""Conduit refresh step for reused visual KV caches on MI355X (gfx950).

The compute lives in the HIP library ``libconduit.so`` behind the C ABI in
``include/conduit.h``; :mod:`.api` is a thin ctypes binding over torch device
tensors.  Importing this package does not load the library; the first call
into :mod:`.api` does, and fails loudly if it is missing.
"""

__all__ = ["api", "workloads"]
