"""Restructured batch normalisation (BN Fission-n-Fusion) for CNN training on
AMD Instinct MI355X (gfx950).

The compute path lives in ``libbnr.so`` (hand-written HIP kernels behind the C
ABI declared in ``include/bnr.h``).  ``paper_1807_01702_amd.bnr`` is the thin
ctypes binding with the same entry-point names; importing this package does
not load the library, so the host-only modules (``synth``) stay usable on a
machine without a GPU.
"""
