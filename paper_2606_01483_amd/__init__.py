"""MI355X-native decode-step attention over a sliding-window-evicted KV cache (Murmur, Section 3.2).

Submodules:
  murmur     -- ctypes binding of libmurmur.so (the C ABI declared in include/murmur.h)
  workloads  -- seeded synthetic inputs shaped like the paper's workloads
  _build     -- hipcc build of libmurmur.so for gfx950

Importing the package loads nothing; ``paper_2606_01483_amd.murmur`` loads the
HIP library and raises if it has not been built.
"""
__all__ = ["murmur", "workloads"]
