"""LoopGuard guarded-decode hot path for AMD Instinct MI355X (gfx950).

Modules:
  lg       ctypes binding of liblg.so (the C ABI in include/lg.h); loading it requires the
           built library and fails loudly without it.
  decoder  GuardedDecoder: device buffers and the per-step call sequence.
  synth    seeded synthetic workloads (inputs only).
  build    compiles liblg.so with hipcc for gfx950.

This package imports nothing at load time so that the input generator can be used without the
HIP library.
"""
