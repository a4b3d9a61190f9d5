"""HilbertA hot path for AMD Instinct MI355X (gfx950).

The compute lives in ``libhilberta.so`` (HIP kernels behind a C ABI, see
``include/hilberta.h``); ``paper_2509_26538_amd.hilberta`` is the thin ctypes
binding with the same function names.  Importing the package loads nothing;
the library is loaded on first use and its absence is an error.
"""

__all__ = ["hilberta", "synth"]
