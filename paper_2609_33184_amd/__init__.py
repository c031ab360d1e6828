"""Chunk-streamed speculative-verification attention for MI355X (gfx950).

The compute path is the C-ABI library ``libspecstream.so`` (hand-written HIP
kernels); ``paper_2609_33184_amd.specstream`` is its ctypes binding.  Importing
this package loads nothing; import the binding explicitly.
"""
