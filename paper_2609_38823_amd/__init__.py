"""MI355X-native (gfx950) hot path of DecoMoE's RCEP MoE layer.

The computation lives in the HIP library ``libdecomoe.so`` (C ABI declared in
``include/decomoe.h``); ``paper_2609_38823_amd.abi`` is a thin ctypes
binding with the same function names, and ``paper_2609_38823_amd.layer``
composes those calls into dense-span and RCEP-span MoE layers.  Importing
the package loads nothing; the library is loaded on first use and the
binding raises if it is missing.
"""
