"""MI355X-native fused bifocal-RoPE attention (Jet-Long, arXiv 2607.07740).

The compute lives in ``libjetlong.so`` (hand-written HIP kernels for gfx950
behind a C ABI declared in ``include/jetlong.h``); ``api`` is a thin ctypes
binding with the same entry-point names.
"""
__all__ = ["api", "synth"]
