"""Scale-QLoRA frozen-code linear layer on MI355X (gfx950).

The compute lives in ``libscaleqlora.so`` (hand-written HIP kernels behind a C
ABI declared in ``include/scaleqlora.h``).  ``paper_2609_04526_amd.sq`` is the
thin ctypes binding with the same entry-point names; it only marshals
arguments (device pointers, sizes, the caller's HIP stream).
"""
