"""KV-Rescue candidate-decode hot path on MI355X (gfx950).

Modules:
  kvr        -- ctypes binding of libkvr (the C ABI in include/kvr.h)
  pipeline   -- per-step decode driver for the synthetic workloads
  workloads  -- the workload shapes (plain data)
  synth      -- seeded synthetic input generators (no method arithmetic)
  build      -- builds libkvr.so in-tree with hipcc for gfx950

The binding is imported lazily so that the generators and workload tables are
usable without a built library.
"""
