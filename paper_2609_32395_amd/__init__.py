"""MI355X-native (gfx950) SMem attention hot path: block-local encoder
attention, joint-softmax reader attention (prefill and batched decode) and a
paged memory-row store with O(b) deletion, behind the C-ABI library
``libsmem.so``.

Importing the package loads nothing; ``paper_2609_32395_amd.smem`` is the
ctypes binding to the library (it fails loudly when the library is missing).
"""
__all__ = ["synth", "smem"]
