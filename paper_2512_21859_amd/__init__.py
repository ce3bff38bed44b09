"""MI355X (gfx950) eviction + decode hot path of TimeBill (arXiv 2512.21859).

The compute lives in libtimebill.so (HIP kernels behind the C ABI in
include/timebill.h); ``_lib`` is its ctypes binding and ``synth`` the seeded
input generators.  Importing the package does not load the library; the
first call into ``_lib`` does, and raises if it has not been built.
"""
from . import synth  # noqa: F401

__all__ = ["synth"]
