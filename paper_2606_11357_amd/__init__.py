"""MI355X-native fused W4A16 / W8A16 weight-only quantized matmul.

The compute path is the HIP library ``libtilefuse.so`` (C ABI in
``include/tilefuse.h``); ``paper_2606_11357_amd.tilefuse`` is its thin ctypes
binding and ``paper_2606_11357_amd.synth`` the seeded input generator.
Importing this package loads nothing; the binding loads the library on first
use and fails loudly if it is not built.
"""
__all__ = ["tilefuse", "synth"]
