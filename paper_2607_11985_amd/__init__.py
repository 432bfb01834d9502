"""MI355X-native batched VQC statevector engine (the execute phase of VQCSim's
compile-once simulation): HIP kernels for gfx950 behind the C ABI of
include/vqc.h.

Submodules
  workloads  seeded circuit structures and inputs (no simulation arithmetic)
  _lib       ctypes binding of libvqc.so (same names as the C ABI)
  api        torch-facing Circuit / VQCFunction (torch supplies memory, streams)
  build      in-tree hipcc build of libvqc.so
"""
