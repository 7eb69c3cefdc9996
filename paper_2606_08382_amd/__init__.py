"""STAR-KV decode attention over a low-rank, quantized KV cache, native to MI355X (gfx950).

The compute path is the C-ABI library ``libstarkv.so`` (hand-written HIP
kernels); ``paper_2606_08382_amd.starkv`` is its ctypes binding.  Importing
this package loads nothing: the library is opened on first use.
"""
__all__ = ["starkv", "synth"]
