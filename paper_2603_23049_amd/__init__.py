"""MI355X-native prefix-reuse prefill (PCR's per-layer KV-reuse hot path).

The product is the C-ABI library ``libpcr.so`` (HIP kernels for gfx950 plus a
host runtime); ``paper_2603_23049_amd.pcr`` is a thin ctypes binding with the
same names. Importing this package loads nothing: the binding is loaded on
first use and raises if the library is missing.
"""
__all__ = ["synth"]
