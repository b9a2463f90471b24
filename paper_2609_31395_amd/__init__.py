"""MI355X (gfx950) library for the compression step of ActKV's action-oriented KV-cache
eviction: score -> select -> compact over a paged KV cache.

Submodules:
  actkv      -- ctypes binding of libactkv.so (the HIP kernels behind the C ABI)
  workloads  -- seeded synthetic inputs (input generation only)
  build      -- compiles libactkv.so with hipcc for gfx950
Importing the package itself loads nothing.
"""
