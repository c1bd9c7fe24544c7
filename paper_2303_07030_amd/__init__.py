"""MI355X-native sparse tensor gradients (nabla-SD hot path).

Submodules:
  nsd      ctypes binding of libnsd (include/nsd.h); importing it requires the
           built library.
  operand  device-resident sparse operands built by the library's builders.
  synth    seeded synthetic workloads (inputs only).
  build    compiles libnsd.so for gfx950.
"""
