"""MI355X (gfx950) attention over a group-wise 4-bit paged KV cache.

The compute path lives in ``libjfkv.so`` (hand-written HIP kernels behind the
C ABI in ``include/jfkv.h``); ``jfkv`` is its ctypes binding and
``workloads`` draws seeded synthetic inputs.  Importing ``jfkv`` fails when the
library has not been built: there is no fallback path.
"""
__all__ = ["jfkv", "workloads"]
