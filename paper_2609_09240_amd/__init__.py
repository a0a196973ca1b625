"""tq — packed ternary GEMV for AMD Instinct MI355X (gfx950).

The compute lives in the C-ABI library ``libtq.so`` (HIP kernels for gfx950,
declared in ``include/tq.h``); ``paper_2609_09240_amd.tq`` is a thin ctypes
binding with the same entry-point names that takes torch tensors for device
memory and streams.  Importing this package loads nothing; the binding loads
the library on first use and raises if it is missing.
"""

__all__ = ["tq", "synth"]
