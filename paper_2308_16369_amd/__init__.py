"""MI355X-native decode-maximal hybrid-batch decoder layer (Sarathi, arXiv 2308.16369).

The compute path lives in ``libsarathi.so`` (hand-written HIP for gfx950,
behind the C-ABI declared in ``include/sarathi.h``); :mod:`.sarathi` is the
thin ctypes binding with the same names.  Importing this package does not
load the library; the first call into the binding does, and fails loudly if
the library is missing.
"""
__all__ = ["sarathi", "accounting"]
