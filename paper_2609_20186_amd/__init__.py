"""SwitchSD speculation-control step for AMD Instinct MI355X (gfx950).

* ``paper_2609_20186_amd.binding``   -- ctypes binding of libswitchsd.so, the
  C ABI declared in include/switchsd.h (n-gram match, probe, switch,
  verify-accept and the fused step);
* ``paper_2609_20186_amd.workloads`` -- seeded synthetic inputs;
* ``paper_2609_20186_amd.build``     -- in-tree build of the HIP library.

The binding is imported on demand so that the input generator works on hosts
without the built library.
"""
__all__ = ["binding", "workloads", "build"]
