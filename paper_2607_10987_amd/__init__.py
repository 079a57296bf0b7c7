"""MI355X-native KV-state operators (materialize, fork, compose, pack/unpack,
attend, evict) over a paged, refcounted block pool.

The compute lives in ``libkvstate.so`` (HIP kernels for gfx950 behind the C ABI
of ``include/kvstate.h``); :mod:`.kvstate` is a thin ctypes binding with the
same function names.  Importing this package loads nothing.
"""
__all__ = ["kvstate"]
