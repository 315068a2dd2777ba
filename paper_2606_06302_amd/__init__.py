"""MI355X-native ragged paged attention for non-uniformly compressed KV caches.

The work runs in libtangram.so (host C++ integer planning + gfx950 HIP
kernels), declared in include/tangram.h.  Submodules:
  tangram  - ctypes binding, one function per C call (import fails loudly if
             the library is not built; there is no fallback path)
  device   - torch plumbing: uploads host tables / plans to device memory
  build    - compiles libtangram.so in-tree
"""
__all__ = ["tangram", "device", "build"]
