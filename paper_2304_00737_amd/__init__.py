"""SparDL sparse-synchronisation hot path for AMD Instinct MI355X (gfx950).

Submodules:
  spardl     -- ctypes binding of libspardl.so (the C ABI in include/spardl.h)
                and a step driver for P simulated workers;
  workloads  -- seeded synthetic gradient generator (input plumbing);
  build      -- in-tree build of the native libraries.
"""

__all__ = ["spardl", "workloads", "build"]
