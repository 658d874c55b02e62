"""CoRun on MI355X: padded fixed-shape batched decode and isolated prefill
with bitwise position invariance, as hand-written HIP kernels for gfx950
behind a C ABI (``include/corun.h``).

Submodules:
  ``corun``     -- the ctypes binding of the C ABI (argument marshalling only)
  ``workload``  -- seeded synthetic inputs (weights, KV contents, batches)
  ``build``     -- compiles ``csrc/`` into ``libcorun.so`` with hipcc

Nothing is loaded at import time; ``corun.load()`` opens the library and
raises if it has not been built.
"""
