"""DriftSched admission hot path on AMD Instinct MI355X (gfx950).

Modules:
  driftsched  binding of the C ABI in include/driftsched.h (loads the HIP
              library; importing it without the built library fails)
  synth       seeded synthetic workloads (input generation only)
  build       compiles the HIP library for gfx950

The binding is not imported here, so the generator can be used on machines
without the built library.
"""
