"""MI355X-native CRVQ hot path: hand-written HIP kernels for gfx950 behind a C ABI.

Submodules:
  crvq      -- ctypes binding of libcrvq.so (argument marshalling only)
  pipeline  -- per-layer quantization as a sequence of library calls
  inputs    -- seeded synthetic workloads (no method arithmetic)
  build     -- hipcc build of libcrvq.so

Importing the package does not load the GPU library; ``crvq.lib()`` does.
"""
