"""Task-guided prefill-time KV-cache eviction (TaskPress, arXiv 2608.03276) on MI355X.

The path is the C-ABI library ``lib/libtaskpress.so`` (HIP kernels for gfx950, sources in
``csrc/``, declarations in ``include/taskpress.h``); ``binding`` is its ctypes binding.
"""
__all__ = ["binding"]
