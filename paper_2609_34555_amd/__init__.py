"""MI355X-native sparse-KV decode hot path (PulseInfer, arXiv 2609.34555).

Submodules:
  pulse      -- ctypes binding of libpulse.so (the gfx950 kernels + C ABI)
  workloads  -- seeded synthetic inputs (no compute of the method)
  harness    -- device buffers of one layer-step built from a workload
"""
