"""MI355X-native statistical plan evaluation (Cornfigurator, arXiv 2512.14098).

The evaluated path runs in hand-written HIP kernels for gfx950 behind the C
ABI declared in ``include/cf.h`` (``libcf.so``); ``paper_2512_14098_amd.cf``
is the thin Python binding (argument marshalling only).  ``inputs`` holds the
seeded synthetic workloads and plan tables.  Importing this package loads
nothing; import ``paper_2512_14098_amd.cf`` to load the library.
"""
__all__ = ["inputs"]
